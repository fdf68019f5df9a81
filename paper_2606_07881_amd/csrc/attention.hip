// Causal multi-head attention, forward and backward, gfx950.
//
// q, k and v live side by side in the fused projection qkv [T, 3d] (head h at
// columns h*dh of each third) and are read in place. Blocks of 64 keys (and
// of 64 or 32 queries) are staged in LDS, and every product is an MFMA chain
// in the convention of device_common.hpp.
//
// Forward (one workgroup per (sequence, head, 64 queries); 4 wavefronts of 16
// queries, heaviest causal blocks first): S^T = K Q^T, so each lane owns one
// query and its per-query statistics stay lane-local. Online softmax runs in
// base 2 with the 1/sqrt(dh) * log2(e) scale folded in. O^T += V^T P^T takes
// P straight from the S^T accumulators (AccPerm order); V^T is staged
// transposed in that same order. The saved statistic is
// lse2 = max + log2(sum), in log2 units of the scaled scores.
//
// Backward: D = rowsum(dO * O) first. Then two kernels recompute P from
// q, k and lse2, so neither needs atomics:
//   dK/dV  (per 64 keys; 16 keys per wavefront):  S = Q K^T and dP = dO V^T
//          with the key in the lane, dV^T += dO^T P, dK^T += Q^T dS;
//   dQ     (per 64 queries; 16 per wavefront):   S^T and dP^T with the query
//          in the lane, dQ^T += K^T dS^T.
#include <type_traits>

#include "device_common.hpp"
#include "kernels.hpp"

namespace paci {
namespace {

constexpr int NT = 256;
constexpr int BKV = 64;   // keys per block
constexpr float LOG2E = 1.4426950408889634f;

// ---------------------------------------------------------------------------------------
template <typename T, int DH, bool DROP>
__global__ void __launch_bounds__(NT) attn_fwd_kernel(const T* qkv, T* out, float* lse2, int S, int H, int d,
                                                       float scale_log2, DropArgs drop) {
  constexpr int V = Vec<T>::V;
  constexpr int BQ = 64;
  constexpr int DKV = DH / V;           // 16-byte vectors per head row
  constexpr int QSTEPS = DH / (4 * V);  // MFMA steps over the head dimension
  constexpr int PSTEPS = BKV / (4 * V); // MFMA steps over a key block
  __shared__ u32x4 sK[DKV * BKV];
  __shared__ u32x4 sVt[(BKV / V) * DH];

  const int nqb = (S + BQ - 1) / BQ;
  const int qb = nqb - 1 - blockIdx.x;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int w = threadIdx.x >> 6, l = lane_id();
  const int64_t ld = 3 * (int64_t)d;
  const T* Qp = qkv + (int64_t)b * S * ld + h * DH;
  const T* Kp = Qp + d;
  const T* Vp = Qp + 2 * d;
  const int q0 = qb * BQ;
  const int qrow = q0 + 16 * w + (l & 15);

  u32x4 qf[QSTEPS];
#pragma unroll
  for (int s = 0; s < QSTEPS; ++s) {
    const int kv = s * 4 + (l >> 4);
    qf[s] = (qrow < S) ? ld16(Qp + (int64_t)qrow * ld + kv * V) : u32x4{0, 0, 0, 0};
  }
  floatx4 acc[DH / 16];
#pragma unroll
  for (int t = 0; t < DH / 16; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const int last_kb = min((q0 + BQ - 1) / BKV, (S - 1) / BKV);
  for (int kb = 0; kb <= last_kb; ++kb) {
    const int k0 = kb * BKV;
    __syncthreads();
    stage_kmajor<T, BKV, DKV, NT>(sK, Kp + (int64_t)k0 * ld, (int)ld, S - k0);
    stage_mnmajor<T, DH, BKV / V, NT>(sVt, Vp + (int64_t)k0 * ld, (int)ld, S - k0, typename AccPerm<T>::type());
    __syncthreads();

    floatx4 st[BKV / 16];
#pragma unroll
    for (int kt = 0; kt < BKV / 16; ++kt) {
      st[kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < QSTEPS; ++s) mma_step<T>(st[kt], lds_frag<BKV>(sK, s, kt * 16), qf[s]);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < BKV / 16; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + kt * 16 + 4 * (l >> 4) + r;
        float x = st[kt][r] * scale_log2;
        if (key > qrow || key >= S) x = -INFINITY;
        st[kt][r] = x;
        mx = fmaxf(mx, x);
      }
    mx = group4_max(mx);
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float rs = 0.f;
#pragma unroll
    for (int kt = 0; kt < BKV / 16; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = exp2f(st[kt][r] - m_use);
        st[kt][r] = p;
        rs += p;
      }
    rs = group4_sum(rs);
    l_run = l_run * alpha + rs;
    m_run = m_new;
    if constexpr (DROP) {   // dropout: the product uses P * keep * scale, the normalizer all of P
#pragma unroll
      for (int kt = 0; kt < BKV / 16; ++kt) {
        const uint32_t bits = drop_row4(drop, bh, qrow, k0 + kt * 16 + 4 * (l >> 4));
#pragma unroll
        for (int r = 0; r < 4; ++r) st[kt][r] = ((bits >> r) & 1) ? st[kt][r] * drop.scale : 0.f;
      }
    }
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) acc[t] *= alpha;
#pragma unroll
    for (int s = 0; s < PSTEPS; ++s) {
      const u32x4 pf = acc_to_frag<T>(st, s);
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) mma_step<T>(acc[t], lds_frag<DH>(sVt, s, t * 16), pf);
    }
  }
  if (qrow < S) {
    const float inv = 1.f / l_run;
    T* op = out + ((int64_t)b * S + qrow) * d + h * DH;
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) {
      const int c = t * 16 + 4 * (l >> 4);
#pragma unroll
      for (int r = 0; r < 4; ++r) op[c + r] = from_f32<T>(acc[t][r] * inv);
    }
    if ((l >> 4) == 0) lse2[(int64_t)bh * S + qrow] = m_run + log2f(l_run);
  }
}

// ---------------------------------------------------------------------------------------
// bf16 kernels on an LDS ring. A block is 64 consecutive rows (keys or
// queries) of one head, [64][dh] bf16, copied by direct-to-LDS loads into a
// ring of NS stages so that the next blocks load while one is used. Row r's
// 16-byte chunk c sits at chunk c ^ blk_swz(r). Fragment reads (ds_read_b128)
// take 16 rows at one chunk per 16 lanes; transpose reads (ds_read_b64_tr_b16)
// take 4 rows x 2 chunks per 16 lanes, two lane groups (8 rows) per cycle. At
// 8 and 16 chunks per row the swizzle sends row bits 0, 2, 1 to chunk bits 0,
// 1, 2 (and row bit 0 also to chunk bit 3 at 16): both kinds of read then hit
// every LDS bank once per cycle, which bank-conflict counters confirm.
template <int CPR> __device__ __forceinline__ int blk_swz(int r) {
  if constexpr (CPR == 4) return (r >> 2) & 3;
  const int f = (r & 1) | (((r >> 2) & 1) << 1) | (((r >> 1) & 1) << 2);
  if constexpr (CPR == 8) return f;
  else return f | ((r & 1) << 3);
}
template <int CPR> __device__ __forceinline__ int blk_slot(int r, int c) { return r * CPR + (c ^ blk_swz<CPR>(r)); }

// MFMA operand: rows = block rows row0 + (l % 16), contracted = head dims of step s.
template <int CPR> __device__ __forceinline__ u32x4 blk_frag(const u32x4* blk, int s, int row0) {
  const int l = lane_id();
  return blk[blk_slot<CPR>(row0 + (l & 15), s * 4 + (l >> 4))];
}
// MFMA operand: rows = head dims dh0 + (l % 16), contracted = the 32 block rows
// of step s in StepPairPerm order (the order acc_to_frag gives accumulators).
template <int CPR> __device__ __forceinline__ u32x4 blk_frag_tr(const u32x4* blk, int s, int dh0) {
  const int l = lane_id(), g = l >> 4, c = l & 15;
  const bf16* base = reinterpret_cast<const bf16*>(blk);
  const int e = dh0 + 4 * (c & 3);
  const int r_lo = s * 32 + 4 * g + (c >> 2), r_hi = r_lo + 16;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(base + blk_slot<CPR>(r_lo, e >> 3) * 8 + (e & 7)));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(base + blk_slot<CPR>(r_hi, e >> 3) * 8 + (e & 7)));
  const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  return u32x4{a[0], a[1], b[0], b[1]};
}
// Issue this thread's loads of one block (rows src[0..63], row stride ld) into
// LDS byte address lds. Rows at or past rows_valid (>= 1) re-read the last
// valid row; every consumer masks those rows out.
template <int CPR, int NT>
__device__ __forceinline__ void blk_fill(const bf16* src, int64_t ld, int rows_valid, uint32_t lds, int w, int l) {
  constexpr int L = 64 * CPR / NT;
  static_assert(L >= 1 && (64 * CPR) % NT == 0, "block slots must split evenly over the threads");
#pragma unroll
  for (int p = 0; p < L; ++p) {
    const int blk = p * (NT / 64) + w;
    const int slot = blk * 64 + l;
    const int r = slot / CPR;
    const int c = (slot % CPR) ^ blk_swz<CPR>(r);
    const int rr = min(r, rows_valid - 1);
    dma16(src + (int64_t)rr * ld + c * 8, lds + (uint32_t)(blk * 1024));
  }
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}

// Forward, bf16: a workgroup takes 64 * QS * 4 queries, each wavefront 16 * QS
// of them (QS sub-tiles of 16, the query in the lane as in the kernel above),
// so every K and V fragment read from LDS feeds QS MFMAs. Key blocks are 64.
template <int DH> struct FwdRing {
  static constexpr int CPR = DH / 8, KS = DH / 32;
  static constexpr int QS = DH == 32 ? 4 : (DH == 64 ? 2 : 1), WAVES = DH == 32 ? 4 : 8, NTF = 64 * WAVES;
  static constexpr int WQ = 16 * QS, BQ = WAVES * WQ;
  // blocks kb (V) and kb + 1 (K) are read in the same iteration, kb + 2 loads
  static constexpr int NS = 4;
  static constexpr int BLK = 64 * CPR;          // 16-byte slots per block
  static constexpr int L = 2 * BLK / NTF;       // loads per thread per stage (K and V)
};

// The key loop is software-pipelined (at head dim 64 and 128): while a
// wavefront runs the online softmax of key block kb on its vector ALUs, the
// MFMAs of the scores of block kb + 1 are interleaved with it, so the matrix
// unit is not idle during the exponentials. A wavefront's queries start at a multiple of 16 * QS, which
// divides 64, so every key block before its last one ends before its first
// query and inside the sequence: only the last block is masked.
template <int DH, bool DROP>
__global__ void __launch_bounds__(FwdRing<DH>::NTF, 2) attn_fwd_ring_kernel(const bf16* qkv, bf16* out, float* lse2, int S, int H,
                                                               int d, float scale_log2, DropArgs drop) {
  using C = FwdRing<DH>;
  constexpr int QS = C::QS, KS = C::KS, NS = C::NS, CPR = C::CPR;
  __shared__ u32x4 ring[NS * 2 * C::BLK];
  const int nqb = (S + C::BQ - 1) / C::BQ;
  const int qb = nqb - 1 - blockIdx.y;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int w = threadIdx.x >> 6, l = lane_id(), g = l >> 4;
  const int wu = __builtin_amdgcn_readfirstlane(w);
  const int64_t ld = 3 * (int64_t)d;
  const bf16* Qp = qkv + (int64_t)b * S * ld + h * DH;
  const bf16* Kp = Qp + d;
  const bf16* Vp = Qp + 2 * d;
  const int q0 = qb * C::BQ, qw0 = q0 + w * C::WQ;
  const uint32_t ring_lds = lds_addr(ring);
  const int nkb = min((q0 + C::BQ - 1) / BKV, (S - 1) / BKV) + 1;
  const int my_last = (qw0 < S) ? min((qw0 + C::WQ - 1) / BKV, (S - 1) / BKV) : -1;

  u32x4 qf[QS][KS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int row = qw0 + 16 * qs + (l & 15);
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qf[qs][s] = (row < S) ? ld16(Qp + (int64_t)row * ld + s * 32 + 8 * g) : u32x4{0, 0, 0, 0};
  }
  floatx4 acc[QS][DH / 16];
  // the softmax normalizer: without dropout an MFMA of the probability
  // fragments against ones (the same bf16 P as the numerator, no cross-lane
  // sums); with dropout a running sum of all of P in fp32
  floatx4 lacc[QS];
  const u32x4 ones = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};   // bf16 1.0 pairs
  float m_run[QS], l_run[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    m_run[qs] = -INFINITY;
    l_run[qs] = 0.f;
    lacc[qs] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) acc[qs][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  auto fill = [&](int kb) {
    const uint32_t st = ring_lds + (uint32_t)((kb % NS) * 2 * C::BLK * 16);
    const int k0 = kb * BKV;
    blk_fill<CPR, C::NTF>(Kp + (int64_t)k0 * ld, ld, S - k0, st, wu, l);
    blk_fill<CPR, C::NTF>(Vp + (int64_t)k0 * ld, ld, S - k0, st + C::BLK * 16, wu, l);
  };
  // raw scores q k^T of key block kb
  auto scores = [&](int kb, floatx4 (&sc)[QS][4]) {
    const u32x4* sK = ring + (kb % NS) * 2 * C::BLK;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      u32x4 kf[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s) kf[s] = blk_frag<CPR>(sK, s, kt * 16);
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) {
        sc[qs][kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) mma_step<bf16>(sc[qs][kt], kf[s], qf[qs][s]);
      }
    }
  };
  // online softmax of block kb's scores: running max and sum, rescaled
  // accumulators, and the probabilities (dropped ones zeroed) as bf16 fragments
  auto softmax = [&](auto masked, int kb, floatx4 (&sc)[QS][4], u32x4 (&pf)[QS][2]) {
    const int k0 = kb * BKV;
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      const int qrow = qw0 + 16 * qs + (l & 15);
      if constexpr (decltype(masked)::value) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = k0 + kt * 16 + 4 * g + r;
            if (key > qrow || key >= S) sc[qs][kt][r] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sc[qs][kt][r]);
      mx = group4_max(mx);
      const float m_new = fmaxf(m_run[qs], mx * scale_log2);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = fast_exp2(m_run[qs] - m_use);
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[qs][kt][r] = fast_exp2(fmaf(sc[qs][kt][r], scale_log2, -m_use));
      if constexpr (DROP) {
        float rs = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) rs += sc[qs][kt][r];
        l_run[qs] = l_run[qs] * alpha + group4_sum(rs);
      } else {
        lacc[qs] *= alpha;
      }
      m_run[qs] = m_new;
      if constexpr (DROP) {   // dropout: the product uses P * keep * scale, the normalizer all of P
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          const uint32_t bits = drop_row4(drop, bh, qrow, k0 + kt * 16 + 4 * g);
#pragma unroll
          for (int r = 0; r < 4; ++r) sc[qs][kt][r] = ((bits >> r) & 1) ? sc[qs][kt][r] * drop.scale : 0.f;
        }
      }
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) acc[qs][t] *= alpha;
      pf[qs][0] = acc_to_frag<bf16>(sc[qs], 0);
      pf[qs][1] = acc_to_frag<bf16>(sc[qs], 1);
    }
  };
  auto pv = [&](int kb, const u32x4 (&pf)[QS][2]) {
    const u32x4* sV = ring + (kb % NS) * 2 * C::BLK + C::BLK;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) {
        const u32x4 vf = blk_frag_tr<CPR>(sV, s, t * 16);
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) mma_step<bf16>(acc[qs][t], vf, pf[qs][s]);
      }
    if constexpr (!DROP) {
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) mma_step<bf16>(lacc[qs], ones, pf[qs][s]);
    }
  };
  // iteration kb: blocks up to min(nkb - 1, kb + NS - 2) have been issued;
  // wait for block kb + 1, whose keys this iteration reads, then refill the
  // stage of block kb - 1, which every wavefront has finished with
  // (at 4 query sub-tiles per wavefront the two score arrays would not fit in
  // registers: that variant reads and computes block kb only)
  constexpr bool PIPE = QS <= 2;
  auto step = [&](int kb, floatx4 (&cur)[QS][4], floatx4 (&nxt)[QS][4]) {
    const int newest = PIPE ? kb + 1 : kb;   // the newest block this iteration reads
    if (newest < nkb) wait_loads<C::L, NS - 2>(min(nkb - 1, kb + NS - 2) - newest);
    wait_lds_reads();
    barrier_no_fence();
    if (kb + NS - 1 < nkb) fill(kb + NS - 1);
    if (kb > my_last) return;
    u32x4 pf[QS][2];
    if constexpr (!PIPE) {
      scores(kb, cur);
      if (kb < my_last) softmax(std::false_type{}, kb, cur, pf);
      else softmax(std::true_type{}, kb, cur, pf);
    } else if (kb < my_last) {
      scores(kb + 1, nxt);
      softmax(std::false_type{}, kb, cur, pf);
      // interleave: the fragment reads first, then one MFMA per few ALU instructions
      __builtin_amdgcn_sched_group_barrier(0x100, 4 * KS, 0);
#pragma unroll
      for (int i = 0; i < 4 * KS * QS; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
      }
    } else {
      softmax(std::true_type{}, kb, cur, pf);
    }
    pv(kb, pf);
  };

#pragma unroll
  for (int t = 0; t < NS - 1; ++t)
    if (t < nkb) fill(t);
  floatx4 sA[QS][4], sB[QS][4];
  // every load so far, the query fragments included, through a wait the
  // compiler sees: it then knows qf has landed and puts no vmcnt(0) in the
  // loop, which would also wait for the ring's prefetches
  wait_vmcnt_all();
  barrier_no_fence();
  if (PIPE && my_last >= 0) scores(0, sA);
  for (int kb = 0; kb < nkb; kb += 2) {
    step(kb, sA, sB);
    if (kb + 1 < nkb) step(kb + 1, sB, sA);
  }
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int qrow = qw0 + 16 * qs + (l & 15);
    if (qrow < S) {
      if constexpr (!DROP) l_run[qs] = lacc[qs][0];   // every row of the product holds the row sum
      const float inv = 1.f / l_run[qs];
      bf16* op = out + ((int64_t)b * S + qrow) * d + h * DH;
#pragma unroll
      for (int t = 0; t < DH / 16; ++t)
        *reinterpret_cast<u32x2*>(op + t * 16 + 4 * g) =
            u32x2{pack_bf16x2(acc[qs][t][0] * inv, acc[qs][t][1] * inv),
                  pack_bf16x2(acc[qs][t][2] * inv, acc[qs][t][3] * inv)};
      if (g == 0) lse2[(int64_t)bh * S + qrow] = m_run[qs] + log2f(l_run[qs]);
    }
  }
}

// D[bh][q] = sum_c dO[q][h*dh + c] * O[q][h*dh + c]; one wavefront per (token, head) row group.
template <typename T, int DH>
__global__ void __launch_bounds__(NT) attn_dsum_kernel(const T* o, const T* dO, float* D, int S, int H, int d,
                                                        int64_t rows) {
  constexpr int V = Vec<T>::V;
  constexpr int LPR = DH / V;  // lanes per (token, head) row
  const int64_t gid = (int64_t)blockIdx.x * NT + threadIdx.x;
  const int64_t row = gid / LPR;  // row = token * H + h
  const int part = gid % LPR;
  float s = 0.f;
  if (row < rows) {
    const int64_t tok = row / H;
    const int h = row % H;
    const int64_t off = tok * d + h * DH + part * V;
    const u32x4 a = ld16(o + off), g = ld16(dO + off);
#pragma unroll
    for (int j = 0; j < V; ++j) s += vget<T>(a, j) * vget<T>(g, j);
  }
#pragma unroll
  for (int w = LPR / 2; w >= 1; w >>= 1) s += __shfl_xor(s, w, 64);
  if (row < rows && part == 0) {
    const int64_t tok = row / H;
    const int h = row % H;
    const int64_t b = tok / S, q = tok % S;
    D[(b * H + h) * S + q] = s;
  }
}

// ---------------------------------------------------------------------------------------
template <typename T, int DH, bool DROP>
__global__ void __launch_bounds__(NT) attn_bwd_dkdv_kernel(const T* qkv, const T* dO, const float* lse2,
                                                            const float* Dsum, T* dqkv, int S, int H, int d,
                                                            float scale_log2, float scale, DropArgs drop) {
  constexpr int V = Vec<T>::V;
  constexpr int BQ = (DH >= 128) ? 32 : 64;  // queries per staged block (LDS budget)
  constexpr int DKV = DH / V;
  constexpr int QSTEPS = DH / (4 * V);
  constexpr int RSTEPS = BQ / (4 * V);       // MFMA steps over a query block
  __shared__ u32x4 sQ[DKV * BQ];
  __shared__ u32x4 sdO[DKV * BQ];
  __shared__ u32x4 sQt[(BQ / V) * DH];
  __shared__ u32x4 sdOt[(BQ / V) * DH];
  __shared__ float sL[BQ], sD[BQ];

  const int kb = blockIdx.x;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int w = threadIdx.x >> 6, l = lane_id();
  const int64_t ld = 3 * (int64_t)d;
  const T* Qp = qkv + (int64_t)b * S * ld + h * DH;
  const T* Kp = Qp + d;
  const T* Vp = Qp + 2 * d;
  const T* dOp = dO + (int64_t)b * S * d + h * DH;
  const float* Lp = lse2 + (int64_t)bh * S;
  const float* Dp = Dsum + (int64_t)bh * S;
  const int k0 = kb * BKV;
  const int key = k0 + 16 * w + (l & 15);

  u32x4 kf[QSTEPS], vf[QSTEPS];
#pragma unroll
  for (int s = 0; s < QSTEPS; ++s) {
    const int kv = s * 4 + (l >> 4);
    kf[s] = (key < S) ? ld16(Kp + (int64_t)key * ld + kv * V) : u32x4{0, 0, 0, 0};
    vf[s] = (key < S) ? ld16(Vp + (int64_t)key * ld + kv * V) : u32x4{0, 0, 0, 0};
  }
  floatx4 adk[DH / 16], adv[DH / 16];
#pragma unroll
  for (int t = 0; t < DH / 16; ++t) adk[t] = adv[t] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int q0 = (k0 / BQ) * BQ; q0 < S; q0 += BQ) {
    __syncthreads();
    stage_kmajor<T, BQ, DKV, NT>(sQ, Qp + (int64_t)q0 * ld, (int)ld, S - q0);
    stage_kmajor<T, BQ, DKV, NT>(sdO, dOp + (int64_t)q0 * d, d, S - q0);
    stage_mnmajor<T, DH, BQ / V, NT>(sQt, Qp + (int64_t)q0 * ld, (int)ld, S - q0, typename AccPerm<T>::type());
    stage_mnmajor<T, DH, BQ / V, NT>(sdOt, dOp + (int64_t)q0 * d, d, S - q0, typename AccPerm<T>::type());
    if (threadIdx.x < BQ) {
      const int q = q0 + threadIdx.x;
      sL[threadIdx.x] = (q < S) ? Lp[q] : 0.f;
      sD[threadIdx.x] = (q < S) ? Dp[q] : 0.f;
    }
    __syncthreads();
    floatx4 P[BQ / 16], dS[BQ / 16];
#pragma unroll
    for (int qt = 0; qt < BQ / 16; ++qt) {
      floatx4 s = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < QSTEPS; ++st) {
        mma_step<T>(s, lds_frag<BQ>(sQ, st, qt * 16), kf[st]);
        mma_step<T>(dp, lds_frag<BQ>(sdO, st, qt * 16), vf[st]);
      }
      const uint32_t bits = DROP ? drop_col4(drop, bh, q0 + qt * 16 + 4 * (l >> 4), key) : 0xfu;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qi = qt * 16 + 4 * (l >> 4) + r;
        const int q = q0 + qi;
        const bool ok = (key <= q) && (q < S) && (key < S);
        const float p = ok ? exp2f(s[r] * scale_log2 - sL[qi]) : 0.f;
        // dropout M = keep * scale: dV takes P M, dP = (dO V^T) M
        const float mk = DROP ? (((bits >> r) & 1) ? drop.scale : 0.f) : 1.f;
        P[qt][r] = p * mk;
        dS[qt][r] = p * (dp[r] * mk - sD[qi]);
      }
    }
#pragma unroll
    for (int st = 0; st < RSTEPS; ++st) {
      const u32x4 pf = acc_to_frag<T>(P, st), sf = acc_to_frag<T>(dS, st);
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) {
        mma_step<T>(adv[t], lds_frag<DH>(sdOt, st, t * 16), pf);
        mma_step<T>(adk[t], lds_frag<DH>(sQt, st, t * 16), sf);
      }
    }
  }
  if (key < S) {
    T* dk = dqkv + ((int64_t)b * S + key) * ld + d + h * DH;
    T* dv = dk + d;
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) {
      const int c = t * 16 + 4 * (l >> 4);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        dk[c + r] = from_f32<T>(adk[t][r] * scale);
        dv[c + r] = from_f32<T>(adv[t][r]);
      }
    }
  }
}

template <typename T, int DH, bool DROP>
__global__ void __launch_bounds__(NT) attn_bwd_dq_kernel(const T* qkv, const T* dO, const float* lse2,
                                                          const float* Dsum, T* dqkv, int S, int H, int d,
                                                          float scale_log2, float scale, DropArgs drop) {
  constexpr int V = Vec<T>::V;
  constexpr int BQ = 64;
  constexpr int DKV = DH / V;
  constexpr int QSTEPS = DH / (4 * V);
  constexpr int PSTEPS = BKV / (4 * V);
  __shared__ u32x4 sK[DKV * BKV];
  __shared__ u32x4 sV[DKV * BKV];
  __shared__ u32x4 sKt[(BKV / V) * DH];

  const int nqb = (S + BQ - 1) / BQ;
  const int qb = nqb - 1 - blockIdx.x;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int w = threadIdx.x >> 6, l = lane_id();
  const int64_t ld = 3 * (int64_t)d;
  const T* Qp = qkv + (int64_t)b * S * ld + h * DH;
  const T* Kp = Qp + d;
  const T* Vp = Qp + 2 * d;
  const T* dOp = dO + (int64_t)b * S * d + h * DH;
  const int q0 = qb * BQ;
  const int qrow = q0 + 16 * w + (l & 15);
  const bool qok = qrow < S;
  const float lq = qok ? lse2[(int64_t)bh * S + qrow] : 0.f;
  const float Dq = qok ? Dsum[(int64_t)bh * S + qrow] : 0.f;

  u32x4 qf[QSTEPS], gf[QSTEPS];
#pragma unroll
  for (int s = 0; s < QSTEPS; ++s) {
    const int kv = s * 4 + (l >> 4);
    qf[s] = qok ? ld16(Qp + (int64_t)qrow * ld + kv * V) : u32x4{0, 0, 0, 0};
    gf[s] = qok ? ld16(dOp + (int64_t)qrow * d + kv * V) : u32x4{0, 0, 0, 0};
  }
  floatx4 adq[DH / 16];
#pragma unroll
  for (int t = 0; t < DH / 16; ++t) adq[t] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int last_kb = min((q0 + BQ - 1) / BKV, (S - 1) / BKV);
  for (int kb = 0; kb <= last_kb; ++kb) {
    const int k0 = kb * BKV;
    __syncthreads();
    stage_kmajor<T, BKV, DKV, NT>(sK, Kp + (int64_t)k0 * ld, (int)ld, S - k0);
    stage_kmajor<T, BKV, DKV, NT>(sV, Vp + (int64_t)k0 * ld, (int)ld, S - k0);
    stage_mnmajor<T, DH, BKV / V, NT>(sKt, Kp + (int64_t)k0 * ld, (int)ld, S - k0, typename AccPerm<T>::type());
    __syncthreads();
    floatx4 dS[BKV / 16];
#pragma unroll
    for (int kt = 0; kt < BKV / 16; ++kt) {
      floatx4 s = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < QSTEPS; ++st) {
        mma_step<T>(s, lds_frag<BKV>(sK, st, kt * 16), qf[st]);
        mma_step<T>(dp, lds_frag<BKV>(sV, st, kt * 16), gf[st]);
      }
      const uint32_t bits = DROP ? drop_row4(drop, bh, qrow, k0 + kt * 16 + 4 * (l >> 4)) : 0xfu;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + kt * 16 + 4 * (l >> 4) + r;
        const bool ok = qok && (key <= qrow) && (key < S);
        const float p = ok ? exp2f(s[r] * scale_log2 - lq) : 0.f;
        const float mk = DROP ? (((bits >> r) & 1) ? drop.scale : 0.f) : 1.f;
        dS[kt][r] = p * (dp[r] * mk - Dq);
      }
    }
#pragma unroll
    for (int st = 0; st < PSTEPS; ++st) {
      const u32x4 sf = acc_to_frag<T>(dS, st);
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) mma_step<T>(adq[t], lds_frag<DH>(sKt, st, t * 16), sf);
    }
  }
  if (qok) {
    T* dq = dqkv + ((int64_t)b * S + qrow) * ld + h * DH;
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) {
      const int c = t * 16 + 4 * (l >> 4);
#pragma unroll
      for (int r = 0; r < 4; ++r) dq[c + r] = from_f32<T>(adq[t][r] * scale);
    }
  }
}

// ---------------------------------------------------------------------------------------
// Backward, bf16. A pre-pass writes (lse2, D) pairs per query into a buffer
// padded to 64 queries per head, so the workgroups can copy them with the
// blocks. Two kinds of workgroup, in one launch, then recompute P from q, k and
// lse2 (no atomics):
//   dK/dV  per 64 * SUB keys of a wavefront (K and V fragments in registers),
//          streaming 64-query blocks of Q, dO and their pairs through the ring:
//          S = Q K^T and dP = dO V^T with the key in the lane, then
//          dV^T += dO^T P and dK^T += Q^T dS, dO^T and Q^T by transpose reads;
//   dQ     per 64 * SUB queries (Q and dO fragments in registers), streaming
//          64-key blocks of K and V: S^T, dP^T with the query in the lane, then
//          dQ^T += K^T dS^T, K^T by transpose reads.
// head_dim 64: workgroups of 4 wavefronts of 32 rows, two per CU. Each has its
// own barrier, so the two wavefronts of a SIMD drift apart and one's softmax
// VALU work overlaps the other's MFMAs (one workgroup of 8 wavefronts per CU
// keeps them in step: 9% slower for dK/dV, 4% for dQ). 128: 8 of 16 rows;
// 32: 4 of 64 rows.
template <int DH> struct BwdRing {
  static constexpr int CPR = DH / 8, KST = DH / 32;
  static constexpr int SUB = DH == 32 ? 4 : (DH == 64 ? 2 : 1), WAVES = DH == 128 ? 8 : 4, NTB = 64 * WAVES;
  static constexpr int OCC = DH == 32 ? 1 : 2;   // wavefronts per SIMD the register budget must allow
  static constexpr int WR = 16 * SUB, BR = WAVES * WR;
  static constexpr int NS = 4;
  static constexpr int BLK = 64 * CPR;
  static constexpr int PAIR_SLOTS = 32;            // 64 (lse2, D) pairs
  static constexpr int STAGE = 2 * BLK + PAIR_SLOTS;
  static constexpr int L = 2 * BLK / NTB;          // block loads per thread per stage (wave 0 adds the pairs)
};

// (lse2, D) pairs: LPR threads per (token, head) row, PAIR_ROWS consecutive
// rows per thread group with all their loads issued first.
constexpr int PAIR_ROWS = 2;
template <int DH>
__global__ void __launch_bounds__(NT) attn_pairs_kernel(const bf16* o, const bf16* dO, const float* lse2, float* pairs,
                                                         int S, int S_pad, int H, int d, int64_t rows) {
  constexpr int LPR = DH / 8;
  const int64_t gid = (int64_t)blockIdx.x * NT + threadIdx.x;
  const int64_t row0 = gid / LPR * PAIR_ROWS;  // row = token * H + h
  const int part = gid % LPR;
  u32x4 a[PAIR_ROWS], g[PAIR_ROWS];
#pragma unroll
  for (int i = 0; i < PAIR_ROWS; ++i) {
    const int64_t row = row0 + i;
    const int64_t off = (row / H) * d + (row % H) * DH + part * 8;
    a[i] = row < rows ? ld16(o + off) : u32x4{0, 0, 0, 0};
    g[i] = row < rows ? ld16(dO + off) : u32x4{0, 0, 0, 0};
  }
#pragma unroll
  for (int i = 0; i < PAIR_ROWS; ++i) {
    const int64_t row = row0 + i;
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += vget<bf16>(a[i], j) * vget<bf16>(g[i], j);
#pragma unroll
    for (int m = LPR / 2; m >= 1; m >>= 1) sum += __shfl_xor(sum, m, 64);
    if (row < rows && part == 0) {
      const int64_t tok = row / H, bq = tok / S, q = tok % S;
      const int64_t bh = bq * H + row % H;
      pairs[(bh * S_pad + q) * 2] = lse2[bh * S + q];
      pairs[(bh * S_pad + q) * 2 + 1] = sum;
    }
  }
  // queries S .. S_pad - 1 of every head: zeros, so that masked products (p = 0) stay finite
  const int npad = S_pad - S;
  const int64_t heads = rows / S;
  if (npad > 0 && gid < heads * npad) {
    const int64_t bh = gid / npad, q = S + gid % npad;
    pairs[(bh * S_pad + q) * 2] = 0.f;
    pairs[(bh * S_pad + q) * 2 + 1] = 0.f;
  }
}

// Column sums of the gradient tiles a workgroup holds, for the bias gradient of
// the qkv projection: lane l holds columns 4 (l >> 4) + r of 16-column tile t,
// for token l & 15; the 16 lanes of equal l >> 4 (one DPP row) are summed with
// row moves, the waves through LDS (red: WAVES * NCOL floats, free for this
// use), and each column goes out as one atomic add to gbias[col(c)].
template <int WAVES, int NCOL, class Col>
__device__ __forceinline__ void colsum_tiles(float (&v)[NCOL / 16][4], float* red, float* gbias, Col col) {
  const int w = threadIdx.x >> 6, l = lane_id(), g = l >> 4;
#pragma unroll
  for (int t = 0; t < NCOL / 16; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) v[t][r] = row_sum16(v[t][r]);
  if ((l & 15) == 0) {
#pragma unroll
    for (int t = 0; t < NCOL / 16; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[w * NCOL + t * 16 + 4 * g + r] = v[t][r];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < NCOL; c += WAVES * 64) {
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < WAVES; ++u) sum += red[u * NCOL + c];
    atomicAdd(gbias + col(c), sum);
  }
}

// dK/dV of key block kb (ring: NS * STAGE slots of LDS)
template <int DH, bool DROP>
__device__ __forceinline__ void dkdv_ring_body(u32x4* ring, int kb, const bf16* qkv, const bf16* dO,
                                               const float* pairs, bf16* dqkv, int S, int S_pad, int H, int d,
                                               float scale_log2, float scale, float* gbias, const DropArgs& drop) {
  using C = BwdRing<DH>;
  constexpr int SUB = C::SUB, KST = C::KST, NS = C::NS, CPR = C::CPR;
  static_assert(NS * C::STAGE * 4 >= C::WAVES * 2 * DH, "LDS for the column sums");
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int w = threadIdx.x >> 6, l = lane_id(), g = l >> 4;
  const int wu = __builtin_amdgcn_readfirstlane(w);
  const int64_t ld = 3 * (int64_t)d;
  const bf16* Qp = qkv + (int64_t)b * S * ld + h * DH;
  const bf16* Kp = Qp + d;
  const bf16* Vp = Qp + 2 * d;
  const bf16* dOp = dO + (int64_t)b * S * d + h * DH;
  const float* Pp = pairs + (int64_t)bh * S_pad * 2;
  const uint32_t ring_lds = lds_addr(ring);
  const int k0 = kb * C::BR, kw0 = k0 + w * C::WR;
  const int nqb = (S + 63) / 64, qb_first = k0 / 64, njobs = nqb - qb_first;
  const int my_first = (kw0 < S) ? kw0 / 64 : nqb;

  u32x4 kf[SUB][KST], vf[SUB][KST];
#pragma unroll
  for (int ks = 0; ks < SUB; ++ks) {
    const int key = kw0 + 16 * ks + (l & 15);
#pragma unroll
    for (int st = 0; st < KST; ++st) {
      kf[ks][st] = (key < S) ? ld16(Kp + (int64_t)key * ld + st * 32 + 8 * g) : u32x4{0, 0, 0, 0};
      vf[ks][st] = (key < S) ? ld16(Vp + (int64_t)key * ld + st * 32 + 8 * g) : u32x4{0, 0, 0, 0};
    }
  }
  floatx4 adk[SUB][DH / 16], adv[SUB][DH / 16];
#pragma unroll
  for (int ks = 0; ks < SUB; ++ks)
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) adk[ks][t] = adv[ks][t] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto fill = [&](int j) {
    const uint32_t st = ring_lds + (uint32_t)((j % NS) * C::STAGE * 16);
    const int q0 = (qb_first + j) * 64;
    blk_fill<CPR, C::NTB>(Qp + (int64_t)q0 * ld, ld, S - q0, st, wu, l);
    blk_fill<CPR, C::NTB>(dOp + (int64_t)q0 * d, d, S - q0, st + C::BLK * 16, wu, l);
    if (wu == 0 && l < C::PAIR_SLOTS) dma16(Pp + (int64_t)q0 * 2 + l * 4, st + 2 * C::BLK * 16);
  };
#pragma unroll
  for (int t = 0; t < NS - 1; ++t)
    if (t < njobs) fill(t);
  wait_vmcnt_all();   // kf and vf known complete: no vmcnt(0) inside the loop
  for (int j = 0; j < njobs; ++j) {
    wait_loads<C::L, NS - 2>(min(njobs - 1, j + NS - 2) - j);
    wait_lds_reads();
    barrier_no_fence();
    if (j + NS - 1 < njobs) fill(j + NS - 1);
    const int qb = qb_first + j;
    if (qb < my_first) continue;
    const u32x4* sQ = ring + (j % NS) * C::STAGE;
    const u32x4* sdO = sQ + C::BLK;
    const float* sP = reinterpret_cast<const float*>(sQ + 2 * C::BLK);
    const int q0 = qb * 64;
    const bool edge = (q0 < kw0 + C::WR - 1) || (q0 + 64 > S) || (kw0 + C::WR > S);
#pragma unroll
    for (int s = 0; s < 2; ++s) {   // 32 queries: tiles 2s and 2s + 1
      floatx4 sc[SUB][2], dp[SUB][2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        u32x4 qfr[KST], gfr[KST];
#pragma unroll
        for (int st = 0; st < KST; ++st) {
          qfr[st] = blk_frag<CPR>(sQ, st, (2 * s + u) * 16);
          gfr[st] = blk_frag<CPR>(sdO, st, (2 * s + u) * 16);
        }
#pragma unroll
        for (int ks = 0; ks < SUB; ++ks) {
          sc[ks][u] = dp[ks][u] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int st = 0; st < KST; ++st) {
            mma_step<bf16>(sc[ks][u], qfr[st], kf[ks][st]);
            mma_step<bf16>(dp[ks][u], gfr[st], vf[ks][st]);
          }
        }
      }
      // P = 2^(s * scale * log2 e - lse2), dS = P (dP - D); masked entries get P = 0.
      // Dropout M = keep * scale: dV takes P M, and dP = (dO V^T) M.
      uint32_t dbits[2][SUB];
      if constexpr (DROP) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int ks = 0; ks < SUB; ++ks)
            dbits[u][ks] = drop_col4(drop, bh, q0 + (2 * s + u) * 16 + 4 * g, kw0 + 16 * ks + (l & 15));
      }
      auto softmax = [&](auto masked) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int qi = (2 * s + u) * 16 + 4 * g + r;
            const float lq = sP[2 * qi], Dq = sP[2 * qi + 1];
#pragma unroll
            for (int ks = 0; ks < SUB; ++ks) {
              float x = fmaf(sc[ks][u][r], scale_log2, -lq);
              if constexpr (decltype(masked)::value) {
                const int key = kw0 + 16 * ks + (l & 15);
                x = (key <= q0 + qi && q0 + qi < S && key < S) ? x : -INFINITY;
              }
              const float p = fast_exp2(x);
              if constexpr (DROP) {
                const float mk = ((dbits[u][ks] >> r) & 1) ? drop.scale : 0.f;
                sc[ks][u][r] = p * mk;
                dp[ks][u][r] = p * (dp[ks][u][r] * mk - Dq);
              } else {
                sc[ks][u][r] = p;
                dp[ks][u][r] = p * (dp[ks][u][r] - Dq);
              }
            }
          }
      };
      if (edge) softmax(std::true_type());
      else softmax(std::false_type());
      u32x4 pfr[SUB], dsf[SUB];
#pragma unroll
      for (int ks = 0; ks < SUB; ++ks) {
        pfr[ks] = acc_to_frag<bf16>(sc[ks], 0);
        dsf[ks] = acc_to_frag<bf16>(dp[ks], 0);
      }
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) {
        const u32x4 gt = blk_frag_tr<CPR>(sdO, s, t * 16), qt = blk_frag_tr<CPR>(sQ, s, t * 16);
#pragma unroll
        for (int ks = 0; ks < SUB; ++ks) {
          mma_step<bf16>(adv[ks][t], gt, pfr[ks]);
          mma_step<bf16>(adk[ks][t], qt, dsf[ks]);
        }
      }
    }
  }
#pragma unroll
  for (int ks = 0; ks < SUB; ++ks) {
    const int key = kw0 + 16 * ks + (l & 15);
    if (key < S) {
      bf16* dk = dqkv + ((int64_t)b * S + key) * ld + d + h * DH;
      bf16* dv = dk + d;
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) {
        *reinterpret_cast<u32x2*>(dk + t * 16 + 4 * g) =
            u32x2{pack_bf16x2(adk[ks][t][0] * scale, adk[ks][t][1] * scale),
                  pack_bf16x2(adk[ks][t][2] * scale, adk[ks][t][3] * scale)};
        *reinterpret_cast<u32x2*>(dv + t * 16 + 4 * g) =
            u32x2{pack_bf16x2(adv[ks][t][0], adv[ks][t][1]), pack_bf16x2(adv[ks][t][2], adv[ks][t][3])};
      }
    }
  }
  if (gbias != nullptr) {   // uniform: G_bqkv += column sums of dK and dV over this workgroup's keys
    float v[2 * DH / 16][4];
#pragma unroll
    for (int t = 0; t < DH / 16; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float sk = 0.f, sv = 0.f;
#pragma unroll
        for (int ks = 0; ks < SUB; ++ks) {
          sk += adk[ks][t][r];
          sv += adv[ks][t][r];
        }
        v[t][r] = sk * scale;
        v[DH / 16 + t][r] = sv;
      }
    __syncthreads();   // every wave is done with the ring
    colsum_tiles<C::WAVES, 2 * DH>(v, reinterpret_cast<float*>(ring), gbias,
                                   [&](int c) { return (c < DH ? d : 2 * d - DH) + h * DH + c; });
  }
}

// dQ of query block nqb - 1 - yb (ring: NS * 2 * BLK slots of LDS)
template <int DH, bool DROP>
__device__ __forceinline__ void dq_ring_body(u32x4* ring, int yb, const bf16* qkv, const bf16* dO,
                                             const float* pairs, bf16* dqkv, int S, int S_pad, int H, int d,
                                             float scale_log2, float scale, float* gbias, const DropArgs& drop) {
  using C = BwdRing<DH>;
  constexpr int SUB = C::SUB, KST = C::KST, NS = C::NS, CPR = C::CPR;
  static_assert(NS * 2 * C::BLK * 4 >= C::WAVES * DH, "LDS for the column sums");
  const int nqb = (S + C::BR - 1) / C::BR;
  const int qb = nqb - 1 - yb;                   // largest queries first: they see the most keys
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int w = threadIdx.x >> 6, l = lane_id(), g = l >> 4;
  const int wu = __builtin_amdgcn_readfirstlane(w);
  const int64_t ld = 3 * (int64_t)d;
  const bf16* Qp = qkv + (int64_t)b * S * ld + h * DH;
  const bf16* Kp = Qp + d;
  const bf16* Vp = Qp + 2 * d;
  const bf16* dOp = dO + (int64_t)b * S * d + h * DH;
  const float* Pp = pairs + (int64_t)bh * S_pad * 2;
  const uint32_t ring_lds = lds_addr(ring);
  const int q0 = qb * C::BR, qw0 = q0 + w * C::WR;
  const int nkb = min((q0 + C::BR - 1) / BKV, (S - 1) / BKV) + 1;
  const int my_last = (qw0 < S) ? min((qw0 + C::WR - 1) / BKV, (S - 1) / BKV) : -1;

  u32x4 qf[SUB][KST], gf[SUB][KST];
  float lq[SUB], Dq[SUB];
#pragma unroll
  for (int qs = 0; qs < SUB; ++qs) {
    const int q = qw0 + 16 * qs + (l & 15);
    const bool ok = q < S;
#pragma unroll
    for (int st = 0; st < KST; ++st) {
      qf[qs][st] = ok ? ld16(Qp + (int64_t)q * ld + st * 32 + 8 * g) : u32x4{0, 0, 0, 0};
      gf[qs][st] = ok ? ld16(dOp + (int64_t)q * d + st * 32 + 8 * g) : u32x4{0, 0, 0, 0};
    }
    lq[qs] = ok ? Pp[2 * q] : 0.f;
    Dq[qs] = ok ? Pp[2 * q + 1] : 0.f;
  }
  floatx4 adq[SUB][DH / 16];
#pragma unroll
  for (int qs = 0; qs < SUB; ++qs)
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) adq[qs][t] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto fill = [&](int kb) {
    const uint32_t st = ring_lds + (uint32_t)((kb % NS) * 2 * C::BLK * 16);
    const int k0 = kb * BKV;
    blk_fill<CPR, C::NTB>(Kp + (int64_t)k0 * ld, ld, S - k0, st, wu, l);
    blk_fill<CPR, C::NTB>(Vp + (int64_t)k0 * ld, ld, S - k0, st + C::BLK * 16, wu, l);
  };
#pragma unroll
  for (int t = 0; t < NS - 1; ++t)
    if (t < nkb) fill(t);
  wait_vmcnt_all();   // qf, gf, lq and Dq known complete: no vmcnt(0) inside the loop
  for (int kb = 0; kb < nkb; ++kb) {
    wait_loads<C::L, NS - 2>(min(nkb - 1, kb + NS - 2) - kb);
    wait_lds_reads();
    barrier_no_fence();
    if (kb + NS - 1 < nkb) fill(kb + NS - 1);
    if (kb > my_last) continue;
    const u32x4* sK = ring + (kb % NS) * 2 * C::BLK;
    const u32x4* sV = sK + C::BLK;
    const int k0 = kb * BKV;
    const bool edge = (k0 + BKV - 1 > qw0) || (k0 + BKV > S) || (qw0 + C::WR > S);
#pragma unroll
    for (int s = 0; s < 2; ++s) {   // 32 keys: tiles 2s and 2s + 1
      floatx4 sc[SUB][2], dp[SUB][2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        u32x4 kfr[KST], vfr[KST];
#pragma unroll
        for (int st = 0; st < KST; ++st) {
          kfr[st] = blk_frag<CPR>(sK, st, (2 * s + u) * 16);
          vfr[st] = blk_frag<CPR>(sV, st, (2 * s + u) * 16);
        }
#pragma unroll
        for (int qs = 0; qs < SUB; ++qs) {
          sc[qs][u] = dp[qs][u] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int st = 0; st < KST; ++st) {
            mma_step<bf16>(sc[qs][u], kfr[st], qf[qs][st]);
            mma_step<bf16>(dp[qs][u], vfr[st], gf[qs][st]);
          }
        }
      }
      auto softmax = [&](auto masked) {
#pragma unroll
        for (int qs = 0; qs < SUB; ++qs) {
          const int q = qw0 + 16 * qs + (l & 15);
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            // dropout M = keep * scale on dP = dO V^T
            const uint32_t bits = DROP ? drop_row4(drop, bh, q, k0 + (2 * s + u) * 16 + 4 * g) : 0xfu;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              float x = fmaf(sc[qs][u][r], scale_log2, -lq[qs]);
              if constexpr (decltype(masked)::value) {
                const int key = k0 + (2 * s + u) * 16 + 4 * g + r;
                x = (key <= q && key < S && q < S) ? x : -INFINITY;
              }
              const float p = fast_exp2(x);
              const float mk = DROP ? (((bits >> r) & 1) ? drop.scale : 0.f) : 1.f;
              dp[qs][u][r] = p * (dp[qs][u][r] * mk - Dq[qs]);
            }
          }
        }
      };
      if (edge) softmax(std::true_type());
      else softmax(std::false_type());
      u32x4 dsf[SUB];
#pragma unroll
      for (int qs = 0; qs < SUB; ++qs) dsf[qs] = acc_to_frag<bf16>(dp[qs], 0);
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) {
        const u32x4 kt = blk_frag_tr<CPR>(sK, s, t * 16);
#pragma unroll
        for (int qs = 0; qs < SUB; ++qs) mma_step<bf16>(adq[qs][t], kt, dsf[qs]);
      }
    }
  }
#pragma unroll
  for (int qs = 0; qs < SUB; ++qs) {
    const int q = qw0 + 16 * qs + (l & 15);
    if (q < S) {
      bf16* dq = dqkv + ((int64_t)b * S + q) * ld + h * DH;
#pragma unroll
      for (int t = 0; t < DH / 16; ++t)
        *reinterpret_cast<u32x2*>(dq + t * 16 + 4 * g) =
            u32x2{pack_bf16x2(adq[qs][t][0] * scale, adq[qs][t][1] * scale),
                  pack_bf16x2(adq[qs][t][2] * scale, adq[qs][t][3] * scale)};
    }
  }
  if (gbias != nullptr) {   // uniform: G_bqkv += column sums of dQ over this workgroup's queries
    float v[DH / 16][4];
#pragma unroll
    for (int t = 0; t < DH / 16; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float sq = 0.f;
#pragma unroll
        for (int qs = 0; qs < SUB; ++qs) sq += adq[qs][t][r];
        v[t][r] = sq * scale;
      }
    __syncthreads();   // every wave is done with the ring
    colsum_tiles<C::WAVES, DH>(v, reinterpret_cast<float*>(ring), gbias, [&](int c) { return h * DH + c; });
  }
}

// The backward kernel: dK/dV and dQ in one launch (grid y below ny: dK/dV of key
// block y, smallest keys first; the rest: dQ, largest queries first), so that
// the tail of the dK/dV blocks overlaps the first dQ blocks and the two share
// CUs (7% faster than two launches at head dim 64).
template <int DH, bool DROP>
__global__ void __launch_bounds__(BwdRing<DH>::NTB, BwdRing<DH>::OCC) attn_bwd_ring_kernel(const bf16* qkv, const bf16* dO, const float* pairs,
                                                               bf16* dqkv, int S, int S_pad, int H, int d,
                                                               float scale_log2, float scale, float* gbias,
                                                               DropArgs drop, int ny) {
  using C = BwdRing<DH>;
  constexpr int SLOTS = C::STAGE > 2 * C::BLK ? C::NS * C::STAGE : C::NS * 2 * C::BLK;
  __shared__ u32x4 ring[SLOTS];
  if ((int)blockIdx.y < ny)
    dkdv_ring_body<DH, DROP>(ring, blockIdx.y, qkv, dO, pairs, dqkv, S, S_pad, H, d, scale_log2, scale, gbias, drop);
  else
    dq_ring_body<DH, DROP>(ring, blockIdx.y - ny, qkv, dO, pairs, dqkv, S, S_pad, H, d, scale_log2, scale, gbias,
                           drop);
}

template <typename T, int DH>
hipError_t fwd_launch(const void* qkv, void* o, float* lse2, int mu, int S, int H, const DropArgs& drop,
                      hipStream_t st) {
  const int d = H * DH;
  const float scale_log2 = LOG2E / sqrtf((float)DH);
  if constexpr (sizeof(T) == 2) {
    using C = FwdRing<DH>;
    dim3 grid(mu * H, (S + C::BQ - 1) / C::BQ);   // x fastest: every head's heaviest query block first
    if (drop.thr)
      hipLaunchKernelGGL((attn_fwd_ring_kernel<DH, true>), grid, dim3(C::NTF), 0, st,
                         reinterpret_cast<const bf16*>(qkv), reinterpret_cast<bf16*>(o), lse2, S, H, d, scale_log2, drop);
    else
      hipLaunchKernelGGL((attn_fwd_ring_kernel<DH, false>), grid, dim3(C::NTF), 0, st,
                         reinterpret_cast<const bf16*>(qkv), reinterpret_cast<bf16*>(o), lse2, S, H, d, scale_log2, drop);
    return hipGetLastError();
  }
  dim3 grid((S + 63) / 64, mu * H);
  if (drop.thr)
    hipLaunchKernelGGL((attn_fwd_kernel<T, DH, true>), grid, dim3(NT), 0, st, reinterpret_cast<const T*>(qkv),
                       reinterpret_cast<T*>(o), lse2, S, H, d, scale_log2, drop);
  else
    hipLaunchKernelGGL((attn_fwd_kernel<T, DH, false>), grid, dim3(NT), 0, st, reinterpret_cast<const T*>(qkv),
                       reinterpret_cast<T*>(o), lse2, S, H, d, scale_log2, drop);
  return hipGetLastError();
}

template <typename T, int DH>
hipError_t bwd_launch(const void* qkv, const void* o, const void* dO, const float* lse2, float* Dbuf, void* dqkv,
                      float* gbias, int mu, int S, int H, const DropArgs& drop, hipStream_t st) {
  const int d = H * DH;
  const float scale = 1.f / sqrtf((float)DH);
  const float scale_log2 = LOG2E * scale;
  if constexpr (sizeof(T) == 2) {
    using C = BwdRing<DH>;
    const int S_pad = (S + 63) / 64 * 64;
    const int64_t rows = (int64_t)mu * S * H;
    const int64_t threads = (rows + PAIR_ROWS - 1) / PAIR_ROWS * (DH / 8);
    const bf16* q = reinterpret_cast<const bf16*>(qkv);
    const bf16* g = reinterpret_cast<const bf16*>(dO);
    bf16* dq = reinterpret_cast<bf16*>(dqkv);
    const int64_t pad_threads = (int64_t)mu * H * (S_pad - S);
    const int64_t grid_threads = threads > pad_threads ? threads : pad_threads;
    hipLaunchKernelGGL((attn_pairs_kernel<DH>), dim3((unsigned)((grid_threads + NT - 1) / NT)), dim3(NT), 0, st,
                       reinterpret_cast<const bf16*>(o), g, lse2, Dbuf, S, S_pad, H, d, rows);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int ny = (S + C::BR - 1) / C::BR;
    const dim3 grid(mu * H, 2 * ny);   // dK/dV blocks, then dQ blocks
    if (drop.thr)
      hipLaunchKernelGGL((attn_bwd_ring_kernel<DH, true>), grid, dim3(C::NTB), 0, st, q, g, Dbuf, dq, S, S_pad, H, d,
                         scale_log2, scale, gbias, drop, ny);
    else
      hipLaunchKernelGGL((attn_bwd_ring_kernel<DH, false>), grid, dim3(C::NTB), 0, st, q, g, Dbuf, dq, S, S_pad, H, d,
                         scale_log2, scale, gbias, drop, ny);
    return hipGetLastError();
  }
  constexpr int LPR = DH / Vec<T>::V;
  const int64_t rows = (int64_t)mu * S * H;
  const int64_t threads = rows * LPR;
  hipLaunchKernelGGL((attn_dsum_kernel<T, DH>), dim3((unsigned)((threads + NT - 1) / NT)), dim3(NT), 0, st,
                     reinterpret_cast<const T*>(o), reinterpret_cast<const T*>(dO), Dbuf, S, H, d, rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  auto dkdv = drop.thr ? attn_bwd_dkdv_kernel<T, DH, true> : attn_bwd_dkdv_kernel<T, DH, false>;
  hipLaunchKernelGGL(dkdv, dim3((S + BKV - 1) / BKV, mu * H), dim3(NT), 0, st,
                     reinterpret_cast<const T*>(qkv), reinterpret_cast<const T*>(dO), lse2, Dbuf,
                     reinterpret_cast<T*>(dqkv), S, H, d, scale_log2, scale, drop);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  auto dqk = drop.thr ? attn_bwd_dq_kernel<T, DH, true> : attn_bwd_dq_kernel<T, DH, false>;
  hipLaunchKernelGGL(dqk, dim3((S + 63) / 64, mu * H), dim3(NT), 0, st,
                     reinterpret_cast<const T*>(qkv), reinterpret_cast<const T*>(dO), lse2, Dbuf,
                     reinterpret_cast<T*>(dqkv), S, H, d, scale_log2, scale, drop);
  e = hipGetLastError();
  if (e != hipSuccess || gbias == nullptr) return e;
  return colsum_acc(sizeof(T) == 2 ? DT_BF16 : DT_F32, dqkv, 3 * d, mu * S, 3 * d, gbias, st);
}

template <typename T>
hipError_t fwd_dh(const void* qkv, void* o, float* lse2, int mu, int S, int H, int dh, const DropArgs& drop,
                  hipStream_t st) {
  switch (dh) {
    case 32: return fwd_launch<T, 32>(qkv, o, lse2, mu, S, H, drop, st);
    case 64: return fwd_launch<T, 64>(qkv, o, lse2, mu, S, H, drop, st);
    case 128:
      // fp32 at head_dim 128 would exceed the 64 KiB LDS budget of these tilings
      if constexpr (sizeof(T) == 2) return fwd_launch<T, 128>(qkv, o, lse2, mu, S, H, drop, st);
      break;
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t bwd_dh(const void* qkv, const void* o, const void* dO, const float* lse2, float* Dbuf, void* dqkv,
                  float* gbias, int mu, int S, int H, int dh, const DropArgs& drop, hipStream_t st) {
  switch (dh) {
    case 32: return bwd_launch<T, 32>(qkv, o, dO, lse2, Dbuf, dqkv, gbias, mu, S, H, drop, st);
    case 64: return bwd_launch<T, 64>(qkv, o, dO, lse2, Dbuf, dqkv, gbias, mu, S, H, drop, st);
    case 128:
      if constexpr (sizeof(T) == 2)
        return bwd_launch<T, 128>(qkv, o, dO, lse2, Dbuf, dqkv, gbias, mu, S, H, drop, st);
      break;
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t attn_fwd(DType dt, const void* qkv, void* o, float* lse2, int mu, int S, int H, int dh, const DropArgs& drop,
                    hipStream_t st) {
  if (mu <= 0 || S <= 0 || H <= 0) return hipErrorInvalidValue;
  if (dt == DT_BF16) return fwd_dh<bf16>(qkv, o, lse2, mu, S, H, dh, drop, st);
  return fwd_dh<float>(qkv, o, lse2, mu, S, H, dh, drop, st);
}

int64_t attn_bwd_workspace_floats(DType dt, int mu, int S, int H) {
  if (dt == DT_BF16) return 2 * (int64_t)mu * H * ((S + 63) / 64 * 64);
  return (int64_t)mu * H * S;
}

hipError_t attn_bwd(DType dt, const void* qkv, const void* o, const void* dO, const float* lse2, float* Dbuf,
                    void* dqkv, float* gbias, int mu, int S, int H, int dh, const DropArgs& drop, hipStream_t st) {
  if (mu <= 0 || S <= 0 || H <= 0) return hipErrorInvalidValue;
  if (dt == DT_BF16) return bwd_dh<bf16>(qkv, o, dO, lse2, Dbuf, dqkv, gbias, mu, S, H, dh, drop, st);
  return bwd_dh<float>(qkv, o, dO, lse2, Dbuf, dqkv, gbias, mu, S, H, dh, drop, st);
}

}  // namespace paci
