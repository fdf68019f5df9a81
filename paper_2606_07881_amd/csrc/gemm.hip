// Matrix-core GEMM for the stage's linear layers (forward, input gradient and
// weight gradient with fused fp32 accumulation), gfx950.
//
// Work decomposition: one 256-thread workgroup (4 wavefronts, 2 x 2) per
// 128 x 128 output tile; each wavefront owns a 64 x 64 sub-tile = 4 x 4 MFMA
// 16 x 16 tiles. The contracted dimension advances in 8-vector slices (64 bf16 or
// 32 fp32 elements), double-buffered in LDS: the global loads of slice k+1 are
// in flight while slice k is multiplied. Operands stored contracted-major
// (K-major) are copied as 16-byte vectors and read as one 16-byte fragment.
// For bf16, operands stored the other way (MN-major: the weight in dX = dY W,
// both activations in dW = dY^T X) are also copied as 16-byte vectors, into a
// [k][rows] layout read with the gfx950 LDS transpose instruction. fp32
// MN-major operands are transposed in registers (4 x 4 blocks).
//
// Tile order is XCD-aware: workgroup w runs on XCD w % 8, so each XCD gets a
// contiguous range of tiles, walked in groups of 8 tile-rows to keep A and B
// panels in that XCD's L2.
#include "device_common.hpp"
#include <cmath>

#include "kernels.hpp"

namespace paci {
namespace {

constexpr int KVN = 8, GROUP_M = 8;

// Tile configuration: a BM x BN output tile per workgroup, WM x WN per wavefront.
template <int BM_, int BN_, int WM_, int WN_>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int WAVES = (BM / WM) * (BN / WN);
  static constexpr int NT = 64 * WAVES;
};

// Register-staged tile loader (global -> registers -> LDS).
// K-major operands and MN-major bf16 operands are copied as 16-byte vectors
// (MN-major bf16 into the [k][ROWS] transpose-read layout); MN-major fp32
// operands are loaded as 4 x 4 blocks and transposed in registers.
template <typename T, int ROWS, bool KMAJ, int NT>
struct TileLoader {
  static constexpr int V = Vec<T>::V;
  static constexpr bool TR = !KMAJ && sizeof(T) == 2;   // transpose-read layout
  static constexpr int ITEMS = (KMAJ || TR) ? ROWS * KVN : (ROWS / V) * KVN;
  static constexpr int PT = (ITEMS + NT - 1) / NT;
  static constexpr int NV = (KMAJ || TR) ? 1 : V;
  u32x4 r[PT][NV];

  // rows [row0, row0+ROWS) of `rows_total`; contracted [k0, k0 + 8V) of k_end.
  __device__ __forceinline__ void load(const T* src, int64_t ld, int row0, int rows_total, int k0, int k_end,
                                       int tid) {
#pragma unroll
    for (int p = 0; p < PT; ++p) {
      const int it = tid + p * NT;
      if ((ITEMS % NT) != 0 && it >= ITEMS) continue;
      if (KMAJ) {
        const int kv = it % KVN, rr = it / KVN;
        const int row = row0 + rr, k = k0 + kv * V;
        u32x4 v = {0, 0, 0, 0};
        if (row < rows_total && k < k_end) {
          v = ld16(src + (int64_t)row * ld + k);
          if (k + V > k_end) v = vmask_tail<T>(v, k_end - k);
        }
        r[p][0] = v;
      } else if (TR) {
        constexpr int CPL = ROWS / V;             // 16-byte chunks per contracted line
        const int c = it % CPL, kk = it / CPL;
        const int k = k0 + kk, rb = row0 + c * V;
        u32x4 v = {0, 0, 0, 0};
        if (k < k_end && rb < rows_total) {
          v = ld16(src + (int64_t)k * ld + rb);
          if (rb + V > rows_total) v = vmask_tail<T>(v, rows_total - rb);
        }
        r[p][0] = v;
      } else {
        const int kv = it % KVN, rr = it / KVN;
        const int rb = row0 + rr * V;
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const int k = k0 + kv * V + j;
          u32x4 v = {0, 0, 0, 0};
          if (k < k_end && rb < rows_total) {
            v = ld16(src + (int64_t)k * ld + rb);
            if (rb + V > rows_total) v = vmask_tail<T>(v, rows_total - rb);
          }
          r[p][j] = v;
        }
      }
    }
  }

  __device__ __forceinline__ void store(u32x4* tile, int tid) const {
#pragma unroll
    for (int p = 0; p < PT; ++p) {
      const int it = tid + p * NT;
      if ((ITEMS % NT) != 0 && it >= ITEMS) continue;
      if (KMAJ) {
        const int kv = it % KVN, rr = it / KVN;
        tile[lds_slot<ROWS>(kv, rr)] = r[p][0];
      } else if (TR) {
        constexpr int CPL = ROWS / V;
        const int c = it % CPL, kk = it / CPL;
        st16(reinterpret_cast<bf16*>(tile) + trt_elem<ROWS>(kk, c * V), r[p][0]);
      } else {
        const int kv = it % KVN, rr = it / KVN;
        u32x4 out[V];
        transpose_block<T>(r[p], out);
#pragma unroll
        for (int i = 0; i < V; ++i) tile[lds_slot<ROWS>(kv, rr * V + i)] = out[i];
      }
    }
  }

  // operand fragment of MFMA step s for the 16 rows starting at row0
  __device__ __forceinline__ static u32x4 frag(const u32x4* tile, int s, int row0) {
    if (TR) return lds_frag_tr<ROWS>(tile, s, row0);
    return lds_frag<ROWS>(tile, s, row0);
  }
};

// GELU, tanh form: gelu(u) = u (1 + tanh z) / 2 with z = c (u + a u^3). Since
// (1 + tanh z) / 2 is the logistic function of 2z, s = 1 / (1 + 2^(-2 z log2 e)),
// it is u s, and its derivative s + 2 c u s (1 - s) (1 + 3 a u^2). One hardware
// exp2 and one reciprocal (about 1 ulp each); s saturates to 0 or 1.
__device__ __forceinline__ float gelu_sig(float u, float u2) {
  const float k = -2.0f * 1.4426950408889634f * 0.7978845608028654f;   // -2 c log2 e
  return __builtin_amdgcn_rcpf(1.0f + fast_exp2(k * u * fmaf(0.044715f, u2, 1.0f)));
}
// The derivative from u, u^2 and s: s + s (1 - s) u (2c + 6ac u^2).
__device__ __forceinline__ float gelu_grad_s(float u, float u2, float sg) {
  constexpr float c2 = 2.0f * 0.7978845608028654f, c6a = 6.0f * 0.044715f * 0.7978845608028654f;
  return fmaf(fmaf(-sg, sg, sg), u * fmaf(c6a, u2, c2), sg);
}
// The FFN up-projection's epilogue keeps gelu'(u) for the backward instead of
// u, the only use of u there: both values then share one exponential and one
// reciprocal, and the down-projection's input gradient only multiplies.
__device__ __forceinline__ void gelu_and_grad(float u, float& g, float& dg) {
  const float u2 = u * u, sg = gelu_sig(u, u2);
  g = u * sg;
  dg = gelu_grad_s(u, u2, sg);
}

// Four consecutive elements [i, i+4) of a T array as floats (one 8- or 16-byte load).
template <typename T> __device__ __forceinline__ void ld4f(const void* p, int64_t i, float* out) {
  const T* q = reinterpret_cast<const T*>(p) + i;
  if (sizeof(T) == 4) {
    const u32x4 v = ld16(q);
#pragma unroll
    for (int j = 0; j < 4; ++j) out[j] = vget<float>(v, j);
  } else {
    const u32x2 v = *reinterpret_cast<const u32x2*>(q);
    const u32x4 w = {v[0], v[1], 0u, 0u};
#pragma unroll
    for (int j = 0; j < 4; ++j) out[j] = vget<bf16>(w, j);
  }
}
template <typename T> __device__ __forceinline__ float ldf(const void* p, int64_t i) {
  return to_f32(reinterpret_cast<const T*>(p)[i]);
}

// Write four consecutive outputs C[m][n .. n+3].
template <typename TO>
__device__ __forceinline__ void store4(TO* C, int64_t idx, const float* v, int nvalid) {
  if (nvalid >= 4) {
    if (sizeof(TO) == 4) {
      st16(C + idx, u32x4{__builtin_bit_cast(uint32_t, v[0]), __builtin_bit_cast(uint32_t, v[1]),
                          __builtin_bit_cast(uint32_t, v[2]), __builtin_bit_cast(uint32_t, v[3])});
    } else {
      *reinterpret_cast<u32x2*>(C + idx) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    }
  } else {
    for (int j = 0; j < nvalid; ++j) C[idx + j] = from_f32<TO>(v[j]);
  }
}

template <typename T, typename TO, int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int m, int n, const floatx4& acc) {
  if (m >= a.M || n >= a.N) return;
  const int nv = min(4, a.N - n);
  if (EPI == EPI_ACC || EPI == EPI_ATOMIC) {
    float* C = reinterpret_cast<float*>(a.C) + (int64_t)m * a.ldc + n;
    if (EPI == EPI_ATOMIC) {
      for (int j = 0; j < nv; ++j) atomicAdd(C + j, acc[j]);
    } else if (nv == 4) {
      u32x4 old = ld16(C);
      float o[4];
      for (int j = 0; j < 4; ++j) {
        const uint32_t w = old[j];
        o[j] = as_float(w) + acc[j];
      }
      store4<float>(reinterpret_cast<float*>(a.C), (int64_t)m * a.ldc + n, o, 4);
    } else {
      for (int j = 0; j < nv; ++j) C[j] += acc[j];
    }
    return;
  }
  float o[4], bias[4] = {0.f, 0.f, 0.f, 0.f}, aux[4] = {0.f, 0.f, 0.f, 0.f};
  constexpr bool HAS_BIAS = EPI == EPI_BIAS || EPI == EPI_BIAS_RES || EPI == EPI_BIAS_GELU;
  constexpr bool HAS_AUX = EPI == EPI_BIAS_RES || EPI == EPI_GELU_GRAD;
  if (nv == 4) {
    if (HAS_BIAS) {
      const u32x4 b = ld16(a.bias + n);
#pragma unroll
      for (int j = 0; j < 4; ++j) bias[j] = vget<float>(b, j);
    }
    if (HAS_AUX) ld4f<T>(a.aux, (int64_t)m * a.ld_aux + n, aux);
  } else {
    for (int j = 0; j < nv; ++j) {
      if (HAS_BIAS) bias[j] = a.bias[n + j];
      if (HAS_AUX) aux[j] = ldf<T>(a.aux, (int64_t)m * a.ld_aux + n + j);
    }
  }
  float g[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float x = acc[j] + bias[j];
    if (EPI == EPI_BIAS_RES) x += aux[j];
    if (EPI == EPI_GELU_GRAD) x *= aux[j];
    if (EPI == EPI_BIAS_GELU) gelu_and_grad(x, g[j], x);
    o[j] = x;
  }
  store4<TO>(reinterpret_cast<TO*>(a.C), (int64_t)m * a.ldc + n, o, nv);
  if (EPI == EPI_BIAS_GELU) store4<TO>(reinterpret_cast<TO*>(a.C2), (int64_t)m * a.ldc + n, g, nv);
}

__device__ __forceinline__ void tile_coords(int pid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int ntiles = tiles_m * tiles_n;
  int logical = pid;
  if ((ntiles & 7) == 0) logical = (pid & 7) * (ntiles >> 3) + (pid >> 3);
  const int group_size = GROUP_M * tiles_n;
  const int first_m = (logical / group_size) * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  const int in_group = logical % group_size;
  tm = first_m + in_group % gm;
  tn = in_group / gm;
}

template <typename T, typename TO, bool AK, bool BK, int EPI, class CF>
__global__ void __launch_bounds__(CF::NT, 1) gemm_kernel(GemmArgs a, int k_per_split) {
  constexpr int BM = CF::BM, BN = CF::BN, WM = CF::WM, WN = CF::WN, NT = CF::NT;
  constexpr int WAVES_N = BN / WN;
  constexpr int V = Vec<T>::V;
  constexpr int BKE = KVN * V;
  __shared__ u32x4 smem[2][(BM + BN) * KVN];
  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;
  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.N + BN - 1) / BN;
  int tm, tn;
  tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int k_begin = blockIdx.y * k_per_split;
  const int k_end = min(a.K, k_begin + k_per_split);
  const int nk = (k_end - k_begin + BKE - 1) / BKE;
  const int wm0 = (w / WAVES_N) * WM, wn0 = (w % WAVES_N) * WN;

  const T* A = reinterpret_cast<const T*>(a.A);
  const T* B = reinterpret_cast<const T*>(a.B);
  TileLoader<T, BM, AK, NT> la;
  TileLoader<T, BN, BK, NT> lb;
  // fp32 MN-major operands load V x V blocks on part of the threads; spread A and B apart
  const int tid_b = (!AK && !BK && sizeof(T) == 4) ? ((tid + NT / 2) % NT) : tid;

  floatx4 acc[WM / 16][WN / 16];
#pragma unroll
  for (int i = 0; i < WM / 16; ++i)
#pragma unroll
    for (int j = 0; j < WN / 16; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (nk > 0) {
    la.load(A, a.lda, m0, a.M, k_begin, k_end, tid);
    lb.load(B, a.ldb, n0, a.N, k_begin, k_end, tid_b);
    la.store(smem[0], tid);
    lb.store(smem[0] + BM * KVN, tid_b);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      const int kn = k_begin + (kt + 1) * BKE;
      la.load(A, a.lda, m0, a.M, kn, k_end, tid);
      lb.load(B, a.ldb, n0, a.N, kn, k_end, tid_b);
    }
    const u32x4* sa = smem[cur];
    const u32x4* sb = smem[cur] + BM * KVN;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      u32x4 yf[WM / 16], xf[WN / 16];
#pragma unroll
      for (int i = 0; i < WM / 16; ++i) yf[i] = TileLoader<T, BM, AK, NT>::frag(sa, s, wm0 + i * 16);
#pragma unroll
      for (int j = 0; j < WN / 16; ++j) xf[j] = TileLoader<T, BN, BK, NT>::frag(sb, s, wn0 + j * 16);
#pragma unroll
      for (int i = 0; i < WM / 16; ++i)
#pragma unroll
        for (int j = 0; j < WN / 16; ++j) mma_step<T>(acc[i][j], xf[j], yf[i]);
    }
    if (kt + 1 < nk) {
      la.store(smem[cur ^ 1], tid);
      lb.store(smem[cur ^ 1] + BM * KVN, tid_b);
    }
    __syncthreads();
  }
  // lane holds C[m][n .. n+3] with m = row (l % 16) of an A tile, n = 4 (l / 16) of a B tile
#pragma unroll
  for (int i = 0; i < WM / 16; ++i)
#pragma unroll
    for (int j = 0; j < WN / 16; ++j)
      epilogue<T, TO, EPI>(a, m0 + wm0 + i * 16 + (l & 15), n0 + wn0 + j * 16 + 4 * (l >> 4), acc[i][j]);
}

// ============================================================================================
// bf16 pipelined kernel: direct-to-LDS loads into an NS-stage ring.
//
// Each 16-byte slot of a tile is filled by global_load_lds_dwordx4. A wave
// instruction fills 64 consecutive slots, so the LDS layouts are chosen to be
// wave-contiguous:
//   K-major   [row][8 vectors of k], vector kv stored at kv ^ ((row >> 1) & 7);
//             8 lanes fetch one 128-byte row segment, and a 16-row fragment
//             read touches 16 distinct bank groups;
//   MN-major  [k][rows] with 16-byte chunk c of line k at c ^ trt_swz(k),
//             read by ds_read_b64_tr_b16 (see lds_frag_tr).
// Slots outside the operand (rows past M or N, k past K) are filled from a
// zero page, so the ring never holds stale data and the k tail sums exactly.
// The loads of tile kt + NS are issued right after the barrier that publishes
// tile kt + 1, into the stage of tile kt, which every wave has read by then.
// ============================================================================================
template <int BM_, int BN_, int WM_, int WN_, int NS_, int OCC_ = 1>
struct PipeTile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, NS = NS_;
  static constexpr int OCC = OCC_;   // wavefronts per SIMD the register budget must allow
  static constexpr int WAVES = (BM / WM) * (BN / WN);
  static constexpr int NT = 64 * WAVES;
  static constexpr int SLOTS_A = BM * 8, SLOTS_B = BN * 8;       // 16-byte slots per tile
  static constexpr int LA = SLOTS_A / NT, LB = SLOTS_B / NT;     // loads per thread per tile
  static constexpr int STAGE_SLOTS = SLOTS_A + SLOTS_B;
  static_assert(SLOTS_A % NT == 0 && SLOTS_B % NT == 0, "tile slots must split evenly over the threads");
  // epilogue staging: PR rows of BN + 4 floats at a time, in the same LDS
  static constexpr int LDC = BN + 4;
  static constexpr int PR = (BM * LDC <= NS * STAGE_SLOTS * 4) ? BM : (BM > 128 ? 128 : BM);
  static constexpr int SMEM_SLOTS = (NS * STAGE_SLOTS > PR * LDC / 4) ? NS * STAGE_SLOTS : PR * LDC / 4;
  static_assert(BM % PR == 0 && PR % WM == 0 && (PR * LDC) % 4 == 0, "epilogue panels must align with wave rows");
};

__device__ __forceinline__ int kmaj_slot(int row, int kv) { return row * 8 + (kv ^ ((row >> 1) & 7)); }

template <int ROWS> __device__ __forceinline__ u32x4 pipe_frag_k(const u32x4* tile, int s, int row0) {
  const int l = lane_id();
  const int row = row0 + (l & 15), kv = s * 4 + (l >> 4);
  return tile[kmaj_slot(row, kv)];
}


// Issue load p (of ROWS * 8 / NT) of this thread's loads of one operand tile
// (ROWS rows x 64 contracted). `tile` is the LDS byte address of the operand's
// part of the stage, `w` the wave index (wave-uniform).
template <int ROWS, bool KMAJ, int NT>
__device__ __forceinline__ void pipe_fill_one(int p, const bf16* src, int64_t ld, int row0, int rows_total, int k0,
                                              int k_end, uint32_t tile, const void* zeros, int w, int l) {
  {
    const int blk = p * (NT / 64) + w;        // wave-uniform block of 64 slots
    const int slot = blk * 64 + l;
    const void* g;
    bool ok;
    if (KMAJ) {
      const int row = slot >> 3;
      const int kv = (slot & 7) ^ ((row >> 1) & 7);
      const int k = k0 + kv * 8;
      ok = (row0 + row < rows_total) && (k < k_end);
      g = src + (int64_t)(row0 + row) * ld + k;
    } else {
      constexpr int CPL = ROWS / 8;
      const int line = slot / CPL;
      const int c = (slot % CPL) ^ trt_swz<ROWS>(line);
      const int k = k0 + line, rb = row0 + c * 8;
      ok = (k < k_end) && (rb < rows_total);
      g = src + (int64_t)k * ld + rb;
    }
    dma16(ok ? g : zeros, tile + (uint32_t)(blk * 64 * 16));
  }
}

// The address of load p of this thread for contracted offset 0 (add k0 for a
// K-major operand, k0 rows for an MN-major one), with its row (K-major) or
// column group (MN-major) clamped into the operand: a clamped row only feeds
// outputs past M or N, which are never stored. Whole k-steps inside K then
// need one address add per load; the last, partial one takes pipe_fill_one,
// which reads the zero page for every slot outside the operand.
template <int ROWS, bool KMAJ, int NT>
__device__ __forceinline__ const bf16* pipe_fill_base(int p, const bf16* src, int64_t ld, int row0, int rows_total,
                                                      int w, int l) {
  const int blk = p * (NT / 64) + w;
  const int slot = blk * 64 + l;
  if (KMAJ) {
    const int row = slot >> 3;
    const int kv = (slot & 7) ^ ((row >> 1) & 7);
    return src + (int64_t)min(row0 + row, rows_total - 1) * ld + kv * 8;
  } else {
    constexpr int CPL = ROWS / 8;
    const int line = slot / CPL;
    const int c = (slot % CPL) ^ trt_swz<ROWS>(line);
    return src + (int64_t)line * ld + min(row0 + c * 8, (rows_total - 1) & ~7);
  }
}

// Output pass of the staged epilogue (every mode but the atomic one). A unit
// is one 16-byte store: 8 bf16 or 4 fp32 columns. Each thread keeps the same
// unit column for all its rows, so the bias is loaded once; the aux rows of
// all passes are loaded before any store, so their latencies overlap.
template <typename TO, int BN, int PR, int NT> struct EpiGeom {
  static constexpr int U = 16 / sizeof(TO), UPR = BN / U, RPI = NT / UPR, P = PR / RPI;
};
// The bf16 aux rows (residual or u) of a one-panel epilogue, loaded before the
// main loop so that their latency hides behind it: the same units staged_out
// gives this thread, one 16-byte load per row; zeros where staged_out will not
// use them (it then loads for itself).
template <typename TO, int BN, int PR, int NT>
__device__ __forceinline__ void prefetch_aux(const GemmArgs& a, int m0, int n0, int tid,
                                             u32x4 (&pre)[EpiGeom<TO, BN, PR, NT>::P]) {
  using G = EpiGeom<TO, BN, PR, NT>;
  static_assert(G::U == 8, "bf16 output units");
  const int n = n0 + (tid % G::UPR) * G::U, r0 = tid / G::UPR;
  const bf16* ap = reinterpret_cast<const bf16*>(a.aux);
  const bool ok = n + G::U <= a.N && a.ld_aux % 8 == 0 && (reinterpret_cast<uintptr_t>(ap) & 15) == 0;
#pragma unroll
  for (int p = 0; p < G::P; ++p) {
    const int m = m0 + r0 + p * G::RPI;
    pre[p] = (ok && m < a.M) ? ld16g(ap + (int64_t)m * a.ld_aux + n) : u32x4{0, 0, 0, 0};
  }
}

// The bias of this thread's output unit, loaded before the main loop as well.
template <typename TO, int BN, int PR, int NT>
__device__ __forceinline__ void prefetch_bias(const GemmArgs& a, int n0, int tid, float (&pb)[16 / sizeof(TO)]) {
  using G = EpiGeom<TO, BN, PR, NT>;
  const int n = n0 + (tid % G::UPR) * G::U;
#pragma unroll
  for (int j = 0; j < G::U; ++j) pb[j] = n + j < a.N ? a.bias[n + j] : 0.f;
}

template <typename TO, int EPI, int BN, int PR, int NT, bool PRE>
__device__ __forceinline__ void staged_out(const GemmArgs& a, const float* cl, int mb, int n0, int tid,
                                           float (&csum)[16 / sizeof(TO)],
                                           const u32x4 (&pre)[EpiGeom<TO, BN, PR, NT>::P],
                                           const float (&pb)[16 / sizeof(TO)]) {
  constexpr int U = 16 / sizeof(TO), UPR = BN / U, RPI = NT / UPR, P = PR / RPI;
  static_assert(NT % UPR == 0 && PR % RPI == 0, "units must tile the panel");
  constexpr int LDC = BN + 4;
  constexpr bool HAS_BIAS = EPI == EPI_BIAS || EPI == EPI_BIAS_RES || EPI == EPI_BIAS_GELU;
  constexpr bool HAS_AUX = EPI == EPI_BIAS_RES || EPI == EPI_GELU_GRAD;   // aux holds bf16 here
  const int cu = tid % UPR, r0 = tid / UPR;
  const int n = n0 + cu * U;
  if (n >= a.N) return;
  const int nv = min(U, a.N - n);
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  const bool vec = nv == U && a.ldc % U == 0 && al16(a.C) && (EPI != EPI_BIAS_GELU || al16(a.C2)) &&
                   (!HAS_AUX || (a.ld_aux % 8 == 0 && al16(a.aux))) && (!HAS_BIAS || al16(a.bias));
  float bias[U];   // prefetched at kernel start (zero past the last column)
#pragma unroll
  for (int j = 0; j < U; ++j) bias[j] = HAS_BIAS ? pb[j] : 0.f;
  // EPI_ACC: every old value of this thread's units is loaded before the
  // first store, so the loads overlap (the compiler cannot order a load past
  // an earlier store to C, which might alias it)
  u32x4 acc_old[EPI == EPI_ACC ? P : 1];
  if constexpr (EPI == EPI_ACC) {
    const float* Cc = reinterpret_cast<const float*>(a.C);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int m = mb + r0 + p * RPI;
      acc_old[p] = (vec && m < a.M) ? ld16g(Cc + (int64_t)m * a.ldc + n) : u32x4{0, 0, 0, 0};
    }
  }
  float aux[P][U];
  if constexpr (HAS_AUX) {
    const bf16* ap = reinterpret_cast<const bf16*>(a.aux);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int m = mb + r0 + p * RPI;
      if (m < a.M) {
        const int64_t off = (int64_t)m * a.ld_aux + n;
        if (PRE && vec) {
#pragma unroll
          for (int j = 0; j < U; ++j) aux[p][j] = vget<bf16>(pre[p], j);
        } else if (vec) {
#pragma unroll
          for (int h = 0; h < U / 8 + (U < 8 ? 1 : 0); ++h) {
            if constexpr (U >= 8) {
              const u32x4 w = ld16g(ap + off + 8 * h);
#pragma unroll
              for (int j = 0; j < 8; ++j) aux[p][8 * h + j] = vget<bf16>(w, j);
            } else {
              const u32x2 w = *reinterpret_cast<const u32x2*>(ap + off);
#pragma unroll
              for (int j = 0; j < U; ++j) {
                const uint32_t word = w[j >> 1];
                aux[p][j] = as_float((j & 1) ? (word & 0xffff0000u) : (word << 16));
              }
            }
          }
        } else {
#pragma unroll
          for (int j = 0; j < U; ++j) aux[p][j] = j < nv ? (float)ap[off + j] : 0.f;
        }
      }
    }
  }
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int r = r0 + p * RPI, m = mb + r;
    if (m >= a.M) continue;
    float o[U], g2[EPI == EPI_BIAS_GELU ? U : 1];
#pragma unroll
    for (int q = 0; q < U / 4; ++q) {
      const floatx4 v = *reinterpret_cast<const floatx4*>(cl + r * LDC + cu * U + 4 * q);
#pragma unroll
      for (int j = 0; j < 4; ++j) o[4 * q + j] = v[j];
    }
    const int64_t off = (int64_t)m * a.ldc + n;
    if constexpr (EPI == EPI_ACC) {
      float* C = reinterpret_cast<float*>(a.C);
      if (vec) {
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] += as_float(acc_old[p][j]);
      } else {
#pragma unroll
        for (int j = 0; j < U; ++j)
          if (j < nv) o[j] += C[off + j];
      }
    } else if constexpr (EPI == EPI_CE_GRAD) {
      const float l = a.row_lse[m];
      const int y = a.row_tgt[m] - n;
#pragma unroll
      for (int j = 0; j < U; ++j) o[j] = a.alpha * (expf(o[j] - l) - (j == y ? 1.f : 0.f));
    } else {
#pragma unroll
      for (int j = 0; j < U; ++j) {
        float x = o[j] + bias[j];
        if constexpr (EPI == EPI_BIAS_RES) x += aux[p][j];
        if constexpr (EPI == EPI_GELU_GRAD) x *= aux[p][j];
        if constexpr (EPI == EPI_BIAS_GELU) gelu_and_grad(x, g2[j], x);
        o[j] = x;
      }
    }
    if (a.colsum != nullptr) {
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (j < nv) csum[j] += o[j];
    }
    if constexpr (sizeof(TO) == 4 && (EPI == EPI_ACC || EPI == EPI_STORE)) {
      if (a.nonfinite != nullptr) {   // uniform
        bool bad = false;
#pragma unroll
        for (int j = 0; j < U; ++j) bad |= (j < nv) && !__builtin_isfinite(o[j]);
        if (bad) *a.nonfinite = 1;
      }
    }
    TO* C = reinterpret_cast<TO*>(a.C);
    if (vec) {
      if constexpr (sizeof(TO) == 2) {
        st16g(C + off, u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                            pack_bf16x2(o[6], o[7])});
      } else {
        st16g(C + off, u32x4{__builtin_bit_cast(uint32_t, o[0]), __builtin_bit_cast(uint32_t, o[1]),
                            __builtin_bit_cast(uint32_t, o[2]), __builtin_bit_cast(uint32_t, o[3])});
      }
    } else {
#pragma unroll
      for (int j = 0; j < U; ++j)
        if (j < nv) C[off + j] = from_f32<TO>(o[j]);
    }
    if constexpr (EPI == EPI_BIAS_GELU) {
      TO* C2 = reinterpret_cast<TO*>(a.C2);
#pragma unroll
      for (int j = 0; j < U; ++j) o[j] = g2[j];
      if (vec) {
        if constexpr (sizeof(TO) == 2)
          st16g(C2 + off, u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                               pack_bf16x2(o[6], o[7])});
        else
          st16g(C2 + off, u32x4{__builtin_bit_cast(uint32_t, o[0]), __builtin_bit_cast(uint32_t, o[1]),
                               __builtin_bit_cast(uint32_t, o[2]), __builtin_bit_cast(uint32_t, o[3])});
      } else {
#pragma unroll
        for (int j = 0; j < U; ++j)
          if (j < nv) C2[off + j] = from_f32<TO>(o[j]);
      }
    }
  }
}

// Cross-entropy row statistics of a staged panel (EPI_CE_STATS): per row and
// 64-column group, the maximum and the sum of exp(x - max) over the valid
// columns, and the target's logit when the group holds it. Consecutive lanes
// take consecutive rows; a full group is read starting at column r mod 64, so
// the 64 lanes of a wavefront hit 64 distinct banks (row stride BN + 4).
template <int BN, int PR, int NT>
__device__ __forceinline__ void ce_stats_panel(const GemmArgs& a, const float* cl, int mb, int n0, int tid) {
  constexpr int LDC = BN + 4, G = BN / 64;
  static_assert(BN % 64 == 0, "64-column groups must tile the block");
  for (int idx = tid; idx < PR * G; idx += NT) {
    const int r = idx % PR, g = idx / PR;
    const int m = mb + r, nb = n0 + 64 * g;
    if (m >= a.M || nb >= a.N) continue;
    const int nv = min(64, a.N - nb);
    const float* row = cl + r * LDC + 64 * g;
    const int rot = nv == 64 ? r : 0;
    float mx = -INFINITY;
    for (int c = 0; c < nv; ++c) mx = fmaxf(mx, row[(c + rot) & 63]);
    float sum = 0.f;
    for (int c = 0; c < nv; ++c) sum += expf(row[(c + rot) & 63] - mx);
    const int64_t q = (int64_t)m * a.ld_part + nb / 64;
    *reinterpret_cast<float2*>(a.ce_part + 2 * q) = make_float2(mx, sum);
    const int y = a.row_tgt[m] - nb;
    if (y >= 0 && y < nv) a.ce_zt[m] = row[y];
  }
}

// Epilogue through LDS. The accumulator tile goes to LDS as fp32 (row stride
// BN + 4 floats, so the 16 rows a wave writes at once fall in distinct banks)
// and is read back with consecutive lanes on consecutive columns: a wave then
// covers whole 256-byte row segments with each store, and each atomic add
// covers 64 consecutive floats. Tiles larger than the ring are done in row
// panels of PR rows.
template <typename TO, int EPI, class CF, bool PRE, int N_I, int N_J>
__device__ __forceinline__ void staged_epilogue(const GemmArgs& a, float* cl, int m0, int n0, int wm0, int wn0,
                                                const floatx4 (&acc)[N_I][N_J],
                                                const u32x4 (&pre)[EpiGeom<TO, CF::BN, CF::PR, CF::NT>::P],
                                                const float (&pb)[16 / sizeof(TO)]) {
  constexpr int BM = CF::BM, BN = CF::BN, NT = CF::NT, LDC = CF::LDC, PR = CF::PR;
  constexpr int U = 16 / sizeof(TO), UPR = BN / U;
  const int tid = threadIdx.x, l = lane_id();
  float csum[U];
#pragma unroll
  for (int j = 0; j < U; ++j) csum[j] = 0.f;
  // bf16 aux rows of a multi-panel epilogue: each panel's are loaded before its
  // staging, so their latency overlaps the staging and its barriers
  constexpr bool PANEL_AUX = (EPI == EPI_BIAS_RES || EPI == EPI_GELU_GRAD) && sizeof(TO) == 2 && !PRE;
#pragma unroll
  for (int p = 0; p < BM / PR; ++p) {
    u32x4 pre_p[PANEL_AUX ? EpiGeom<TO, BN, PR, NT>::P : 1];
    if constexpr (PANEL_AUX) prefetch_aux<TO, BN, PR, NT>(a, m0 + p * PR, n0, tid, pre_p);
    __syncthreads();   // every wave is done with the ring (or with the previous panel)
    if (wm0 >= p * PR && wm0 < (p + 1) * PR) {
#pragma unroll
      for (int i = 0; i < N_I; ++i)
#pragma unroll
        for (int j = 0; j < N_J; ++j)
          *reinterpret_cast<floatx4*>(cl + (wm0 - p * PR + i * 16 + (l & 15)) * LDC + wn0 + j * 16 + 4 * (l >> 4)) =
              acc[i][j];
    }
    __syncthreads();
    const int mb = m0 + p * PR;
    if constexpr (EPI == EPI_CE_STATS) {
      ce_stats_panel<BN, PR, NT>(a, cl, mb, n0, tid);
    } else if constexpr (EPI == EPI_ATOMIC) {
      float* C = reinterpret_cast<float*>(a.C);
      for (int idx = tid; idx < PR * BN; idx += NT) {
        const int r = idx / BN, c = idx % BN;
        const int m = mb + r, n = n0 + c;
        if (m < a.M && n < a.N) atomicAdd(C + (int64_t)m * a.ldc + n, cl[r * LDC + c]);
      }
    } else {
      if constexpr (PANEL_AUX) staged_out<TO, EPI, BN, PR, NT, true>(a, cl, mb, n0, tid, csum, pre_p, pb);
      else staged_out<TO, EPI, BN, PR, NT, PRE>(a, cl, mb, n0, tid, csum, pre, pb);
    }
  }
  if constexpr (EPI != EPI_ATOMIC && EPI != EPI_CE_STATS && UPR <= 64 && 64 % UPR == 0) {
    if (a.colsum != nullptr) {   // uniform: column sums of the tile's output into a.colsum
      // threads with equal tid % UPR hold the same columns: lanes l, l ^ UPR, ... within a
      // wavefront, then the wavefronts through LDS, then one atomic per column
#pragma unroll
      for (int j = 0; j < U; ++j)
#pragma unroll
        for (int off = UPR; off < 64; off *= 2) csum[j] += __shfl_xor(csum[j], off, 64);
      __syncthreads();   // every thread is done reading the staged tile
      const int w = tid >> 6;
      if (l < UPR) {
#pragma unroll
        for (int j = 0; j < U; ++j) cl[w * BN + l * U + j] = csum[j];
      }
      __syncthreads();
      for (int c = tid; c < BN; c += NT) {
        float sum = 0.f;
#pragma unroll
        for (int v = 0; v < NT / 64; ++v) sum += cl[v * BN + c];
        if (n0 + c < a.N) atomicAdd(a.colsum + n0 + c, sum);
      }
    }
  }
}

// Scheduling pattern for one MFMA step: NREAD LDS reads (of the next step)
// spread evenly between NMFMA independent MFMAs (of this step).
template <int NREAD, int NMFMA>
__device__ __forceinline__ void interleave_reads() {
  constexpr int PER = NMFMA / NREAD > 0 ? NMFMA / NREAD : 1;
#pragma unroll
  for (int i = 0; i < NREAD; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one DS read
    __builtin_amdgcn_sched_group_barrier(0x008, PER, 0); // PER MFMAs
  }
}

template <typename TO, bool AK, bool BK, int EPI, class CF, bool GRP = false>
__global__ void __launch_bounds__(CF::NT, CF::OCC) gemm_pipe_kernel(GemmArgs a, int k_per_split) {
  constexpr int BM = CF::BM, BN = CF::BN, WM = CF::WM, WN = CF::WN, NT = CF::NT, NS = CF::NS;
  constexpr int WAVES_N = BN / WN;
  constexpr int BKE = 64;
  constexpr int L = CF::LA + CF::LB;
  __shared__ u32x4 smem[CF::SMEM_SLOTS];
  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;
  int pid = blockIdx.x;
  int xcd_m = 0;   // grouped weight gradients: XCD blocks of the tile grid (0: generic order)
  if constexpr (GRP) {
    // grouped weight gradients: find this workgroup's problem (wave-uniform scalar loads)
    int p = 0;
    while (p + 1 < a.group_n && pid >= a.group[p + 1].tile0) ++p;
    const WgradProblem& pr = a.group[p];
    pid -= pr.tile0;
    const int tm_all = (pr.M + BM - 1) / BM, tn_all = (pr.N + BN - 1) / BN;
    if (pid >= tm_all * tn_all) return;   // padding to a multiple of 8
    xcd_m = pr.xcd_m;
    a.A = pr.A;
    a.B = pr.B;
    a.C = pr.C;
    a.M = pr.M;
    a.N = pr.N;
    a.lda = pr.M;
    a.ldb = pr.N;
    a.ldc = pr.N;
  }
  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.N + BN - 1) / BN;
  int tm, tn;
  if (xcd_m > 0) {
    // XCD x = pid % 8 takes block (x % xcd_m, x / xcd_m) of bm x bn tiles, column by column
    const int x = pid & 7, k = pid >> 3;
    const int bm = tiles_m / xcd_m, bn = tiles_n / (8 / xcd_m);
    tm = (x % xcd_m) * bm + k % bm;
    tn = (x / xcd_m) * bn + k / bm;
  } else {
    tile_coords(pid, tiles_m, tiles_n, tm, tn);
  }
  const int m0 = tm * BM, n0 = tn * BN;
  const int k_begin = blockIdx.y * k_per_split;
  const int k_end = min(a.K, k_begin + k_per_split);
  const int nk = (k_end - k_begin + BKE - 1) / BKE;
  const int wm0 = (w / WAVES_N) * WM, wn0 = (w % WAVES_N) * WN;
  const bf16* A = reinterpret_cast<const bf16*>(a.A);
  const bf16* B = reinterpret_cast<const bf16*>(a.B);

  const uint32_t smem_lds = (uint32_t)(uintptr_t)((__attribute__((address_space(3))) u32x4*)smem);
  const int wu = __builtin_amdgcn_readfirstlane(w);
  // Per-thread load addresses at contracted offset 0. When every k-step lies
  // wholly inside K, a load is one address add (kf: true; a segmented B adds
  // its segment's offset, one per k-step); fills past the last k-step then
  // repeat the last one's addresses, into stages that are never read.
  // Otherwise each load masks itself against K and the operand (pipe_fill_one).
  const bool kfull = k_end - k_begin >= BKE && (k_end - k_begin) % BKE == 0;   // uniform
  const bf16* fa[CF::LA];
  const bf16* fb[CF::LB];
#pragma unroll
  for (int p = 0; p < CF::LA; ++p) fa[p] = pipe_fill_base<BM, AK, NT>(p, A, a.lda, m0, a.M, wu, l);
#pragma unroll
  for (int p = 0; p < CF::LB; ++p) fb[p] = pipe_fill_base<BN, BK, NT>(p, B, a.ldb, n0, a.N, wu, l);
  // load p of the L loads of tile kt (the A operand's first, then B's)
  auto fill_one = [&](auto kf, int kt, int stage, int p) {   // stage = kt % NS
    const uint32_t st = smem_lds + (uint32_t)(stage * CF::STAGE_SLOTS * 16);
    const int k0 = k_begin + kt * BKE;
    if constexpr (decltype(kf)::value) {
      const int kc = min(k0, k_end - BKE);
      if (p < CF::LA) {
        const int blk = p * (NT / 64) + wu;
        dma16(fa[p] + (AK ? (int64_t)kc : (int64_t)kc * a.lda), st + (uint32_t)(blk * 64 * 16));
      } else {
        const int q = p - CF::LA, blk = q * (NT / 64) + wu;
        int64_t off = BK ? (int64_t)kc : (int64_t)kc * a.ldb;
        if constexpr (!AK && !BK) {
          if (a.seg_rows > 0) {   // uniform: row kc of the window is row kc - sg * seg_rows of segment sg
            const int sg = kc / (int)a.seg_rows;
            off = (int64_t)((a.seg_first + sg) % a.seg_count) * a.seg_stride +
                  (int64_t)(kc - sg * (int)a.seg_rows) * a.ldb;
          }
        }
        dma16(fb[q] + off, st + CF::SLOTS_A * 16 + (uint32_t)(blk * 64 * 16));
      }
    } else if (p < CF::LA) {
      pipe_fill_one<BM, AK, NT>(p, A, a.lda, m0, a.M, k0, k_end, st, a.zeros, wu, l);
    } else if constexpr (!AK && !BK) {
      // weight gradients: B may come in segments of seg_rows contracted rows
      // (a tile never straddles two); past k_end the rows are masked as usual
      const bf16* Bs = B;
      int kb = k0, ke = k_end;
      if (a.seg_rows > 0) {
        const int sg = k0 / (int)a.seg_rows;
        Bs = B + (int64_t)((a.seg_first + sg) % a.seg_count) * a.seg_stride;
        kb = k0 - sg * (int)a.seg_rows;
        ke = k_end - sg * (int)a.seg_rows;
      }
      pipe_fill_one<BN, BK, NT>(p - CF::LA, Bs, a.ldb, n0, a.N, kb, ke, st + CF::SLOTS_A * 16, a.zeros, wu, l);
    } else {
      pipe_fill_one<BN, BK, NT>(p - CF::LA, B, a.ldb, n0, a.N, k0, k_end, st + CF::SLOTS_A * 16, a.zeros, wu, l);
    }
  };
  auto fill = [&](auto kf, int kt, int stage) {
#pragma unroll
    for (int p = 0; p < L; ++p) fill_one(kf, kt, stage, p);
  };

  floatx4 acc[WM / 16][WN / 16];
#pragma unroll
  for (int i = 0; i < WM / 16; ++i)
#pragma unroll
    for (int j = 0; j < WN / 16; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  // bf16 residual or u rows of a one-panel epilogue: loaded now, used after the loop
  constexpr bool PRE = (EPI == EPI_BIAS_RES || EPI == EPI_GELU_GRAD) && sizeof(TO) == 2 && CF::PR == BM;
  u32x4 pre[EpiGeom<TO, BN, CF::PR, NT>::P];
  if constexpr (PRE) prefetch_aux<TO, BN, CF::PR, NT>(a, m0, n0, tid, pre);
  float pb[16 / sizeof(TO)];
  // (tall wave tiles load it after the loop: their registers are taken by the fragments)
  constexpr bool HAS_BIAS = EPI == EPI_BIAS || EPI == EPI_BIAS_RES || EPI == EPI_BIAS_GELU;
  constexpr bool TALL = WM / 16 >= 8;
  if constexpr (HAS_BIAS && !TALL) prefetch_bias<TO, BN, CF::PR, NT>(a, n0, tid, pb);

  // Fragments are double-buffered in registers: the LDS reads of the next
  // MFMA step are issued before the MFMAs of the current one. The barrier that
  // publishes tile kt + 1 sits between the two steps of tile kt; each wave
  // first waits for its own reads of tile kt, so after the barrier the stage of
  // tile kt is free and is refilled at once with tile kt + NS. Loads of a tile
  // are thus issued NS - 1 tiles of MFMA work before they are needed.
  u32x4 ya[WM / 16], xa[WN / 16], yb[WM / 16], xb[WN / 16];
  // MN-major operands: each fragment's transpose-read offset within its tile,
  // computed once (the swizzle makes it a non-affine function of the fragment)
  uint32_t tro_a[WM / 16], tro_b[WN / 16];
#pragma unroll
  for (int i = 0; i < WM / 16; ++i) tro_a[i] = AK ? 0u : lds_frag_tr_off<BM>(wm0 + i * 16);
#pragma unroll
  for (int j = 0; j < WN / 16; ++j) tro_b[j] = BK ? 0u : lds_frag_tr_off<BN>(wn0 + j * 16);
  // stage st (0 .. NS - 1) of the ring; the loop keeps st of k-steps kt and kt + 1
  auto read_step = [&](int st, int s, u32x4* yf, u32x4* xf) {
    const u32x4* sa = smem + st * CF::STAGE_SLOTS;
    const u32x4* sb = sa + CF::SLOTS_A;
    const uint32_t la = smem_lds + (uint32_t)(st * CF::STAGE_SLOTS * 16), lb = la + CF::SLOTS_A * 16;
#pragma unroll
    for (int i = 0; i < WM / 16; ++i)
      yf[i] = AK ? pipe_frag_k<BM>(sa, s, wm0 + i * 16) : lds_frag_tr_at<BM>(la + tro_a[i], s);
#pragma unroll
    for (int j = 0; j < WN / 16; ++j)
      xf[j] = BK ? pipe_frag_k<BN>(sb, s, wn0 + j * 16) : lds_frag_tr_at<BN>(lb + tro_b[j], s);
  };
  auto mma_all = [&](const u32x4* yf, const u32x4* xf) {
#pragma unroll
    for (int i = 0; i < WM / 16; ++i)
#pragma unroll
      for (int j = 0; j < WN / 16; ++j) mma_step<bf16>(acc[i][j], xf[j], yf[i]);
  };
  // fragment f of step s (A's fragments first, then B's), and MFMA q of a step
  auto read_frag = [&](int st, int s, int f, u32x4* yf, u32x4* xf) {
    const u32x4* sa = smem + st * CF::STAGE_SLOTS;
    const u32x4* sb = sa + CF::SLOTS_A;
    const uint32_t la = smem_lds + (uint32_t)(st * CF::STAGE_SLOTS * 16), lb = la + CF::SLOTS_A * 16;
    if (f < WM / 16) yf[f] = AK ? pipe_frag_k<BM>(sa, s, wm0 + f * 16) : lds_frag_tr_at<BM>(la + tro_a[f], s);
    else {
      const int j = f - WM / 16;
      xf[j] = BK ? pipe_frag_k<BN>(sb, s, wn0 + j * 16) : lds_frag_tr_at<BN>(lb + tro_b[j], s);
    }
  };
  auto mma_one = [&](int q, const u32x4* yf, const u32x4* xf) {
    const int i = q / (WN / 16), j = q % (WN / 16);
    mma_step<bf16>(acc[i][j], xf[j], yf[i]);
  };

  // The loop body has no branches: fills past the last tile read the zero page
  // and the reads after the last tile are discarded. Within each MFMA step the
  // scheduler spreads the LDS reads of the next step between the MFMAs.
  constexpr int NRI = (AK ? 1 : 2) * (WM / 16) + (BK ? 1 : 2) * (WN / 16);   // LDS read instructions per step
  constexpr int NM = (WM / 16) * (WN / 16);                                 // MFMAs per step
  constexpr int NF = WM / 16 + WN / 16;                                      // fragments per step
  // weight gradients (both operands MN-major, two workgroups per CU): raise the
  // wave's issue priority over its MFMA steps (measured 1.3% faster there,
  // slightly slower for the K-major products)
  constexpr bool PRIO = !AK && !BK;
  auto main_loop = [&](auto kf) {
#pragma unroll
    for (int t = 0; t < NS; ++t) fill(kf, t, t);
    wait_vmcnt<L * (NS - 1)>();
    barrier_no_fence();
    read_step(0, 0, ya, xa);
    int st0 = 0;   // ring stage of k-step kt
    for (int kt = 0; kt < nk; ++kt) {
      const int st1 = st0 + 1 == NS ? 0 : st0 + 1;   // of k-step kt + 1
      wait_lds_reads();     // reads of ya/xa, issued one MFMA step ago
      if constexpr (PRIO) __builtin_amdgcn_s_setprio(1);
      read_step(st0, 1, yb, xb);
      mma_all(ya, xa);
      interleave_reads<NRI, NM>();
      if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
      wait_lds_reads();     // reads of yb/xb
      wait_vmcnt<L * (NS - 2)>();   // tile kt + 1 has landed; kt + 2 .. kt + NS - 1 may be in flight
      barrier_no_fence();
      // Refill the stage of tile kt (every wave has read it) with tile kt + NS,
      // one load at a time between the MFMAs of this step and the reads of
      // the next: the loads of all waves of the CU reach the address unit
      // spread over the step instead of in one burst that holds up the MFMAs
      // (measured faster with every layout once a load is one address add; the
      // weight gradients also raise the wave's issue priority over the step).
      if constexpr (PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int p = 0; p < L; ++p) {
        fill_one(kf, kt + NS, st0, p);   // tile kt + NS reuses the stage of tile kt
#pragma unroll
        for (int f = p * NF / L; f < (p + 1) * NF / L; ++f) read_frag(st1, 0, f, ya, xa);
#pragma unroll
        for (int q = p * NM / L; q < (p + 1) * NM / L; ++q) mma_one(q, yb, xb);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
      st0 = st1;
    }
  };
  // Tall wave tiles (WM = 128: eight A fragments per step, 128 accumulator
  // VGPRs) fit two wavefronts per SIMD only with the A fragments single-
  // buffered: each is re-read for the next step right after its row's MFMAs
  // have issued, so its register is reused (B stays double-buffered). The
  // ring, barriers and waits are those of the loop above; the refill loads
  // are spread one or more per A row.
  constexpr int G = WM / 16;
  auto main_loop_tall = [&](auto kf) {
#pragma unroll
    for (int t = 0; t < NS; ++t) fill(kf, t, t);
    wait_vmcnt<L * (NS - 1)>();
    barrier_no_fence();
    read_step(0, 0, ya, xa);
    int st0 = 0;
    for (int kt = 0; kt < nk; ++kt) {
      const int st1 = st0 + 1 == NS ? 0 : st0 + 1;
      wait_lds_reads();   // ya/xa of step 0 of tile kt
#pragma unroll
      for (int j = 0; j < WN / 16; ++j) read_frag(st0, 1, G + j, ya, xb);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < G; ++i) {
#pragma unroll
        for (int j = 0; j < WN / 16; ++j) mma_step<bf16>(acc[i][j], xa[j], ya[i]);
        read_frag(st0, 1, i, ya, xb);
        __builtin_amdgcn_sched_barrier(0);
      }
      wait_lds_reads();   // ya/xb of step 1
      wait_vmcnt<L * (NS - 2)>();
      barrier_no_fence();
#pragma unroll
      for (int j = 0; j < WN / 16; ++j) read_frag(st1, 0, G + j, ya, xa);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < G; ++i) {
#pragma unroll
        for (int p = i * L / G; p < (i + 1) * L / G; ++p) fill_one(kf, kt + NS, st0, p);
#pragma unroll
        for (int j = 0; j < WN / 16; ++j) mma_step<bf16>(acc[i][j], xb[j], ya[i]);
        read_frag(st1, 0, i, ya, xa);
        __builtin_amdgcn_sched_barrier(0);
      }
      st0 = st1;
    }
  };
  if constexpr (TALL) {
    if (kfull) main_loop_tall(std::true_type{});
    else main_loop_tall(std::false_type{});
  } else {
    if (kfull) main_loop(std::true_type{});
    else main_loop(std::false_type{});
  }
  wait_vmcnt<0>();   // the fills past the last tile, before the ring is reused
  if constexpr (HAS_BIAS && TALL) prefetch_bias<TO, BN, CF::PR, NT>(a, n0, tid, pb);
  staged_epilogue<TO, EPI, CF, PRE>(a, reinterpret_cast<float*>(smem), m0, n0, wm0, wn0, acc, pre, pb);
}

// Tile configurations; the choice per call is made in launch().
typedef Tile<128, 128, 64, 64> T128x128;

int g_tile_override = -1;  // testing hook: force one configuration

typedef PipeTile<256, 128, 64, 64, 3> P256x128;
typedef PipeTile<128, 128, 64, 64, 4> P128x128;
typedef PipeTile<128, 256, 64, 64, 3> P128x256;
typedef PipeTile<128, 128, 64, 64, 2, 2> P128x128o2;   // two workgroups per CU
// 256 x 256 in eight 128 x 64 wave tiles, two-stage ring (128 KB): a quarter
// fewer LDS reads and a third fewer global -> LDS bytes per FLOP than 256 x 128
typedef PipeTile<256, 256, 128, 64, 2> P256x256;

template <typename TO, bool AK, bool BK, int EPI, class CF>
hipError_t launch_pipe(const GemmArgs& a, int splits, hipStream_t st) {
  constexpr int BKE = 64;
  const int tiles = ((a.M + CF::BM - 1) / CF::BM) * ((a.N + CF::BN - 1) / CF::BN);
  int kps = (a.K + splits - 1) / splits;
  kps = ((kps + BKE - 1) / BKE) * BKE;
  const int used = (a.K + kps - 1) / kps;
  hipLaunchKernelGGL((gemm_pipe_kernel<TO, AK, BK, EPI, CF>), dim3(tiles, used), dim3(CF::NT), 0, st, a, kps);
  return hipGetLastError();
}

int cu_count() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) ==
                                                hipSuccess && n > 0)
      cus = n;
    else
      cus = 256;
  }
  return cus;
}

template <typename T, typename TO, bool AK, bool BK, int EPI, class CF>
hipError_t launch_cf(const GemmArgs& a, int splits, hipStream_t st) {
  constexpr int BKE = KVN * Vec<T>::V;
  const int tiles = ((a.M + CF::BM - 1) / CF::BM) * ((a.N + CF::BN - 1) / CF::BN);
  int kps = (a.K + splits - 1) / splits;
  kps = ((kps + BKE - 1) / BKE) * BKE;
  const int used = (a.K + kps - 1) / kps;
  hipLaunchKernelGGL((gemm_kernel<T, TO, AK, BK, EPI, CF>), dim3(tiles, used), dim3(CF::NT), 0, st, a, kps);
  return hipGetLastError();
}

// The pipelined kernel moves whole 16-byte chunks of 8 elements from global
// memory to LDS, so every chunk must be aligned and lie wholly inside or wholly
// outside the operand: 16-byte aligned bases, leading dimensions and K (and the
// contiguous M or N of an MN-major operand) multiples of 8. Other calls take
// the register-staged kernel, which masks partial vectors.
template <bool AK, bool BK>
bool pipe_eligible(const GemmArgs& a) {
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  return a.zeros != nullptr && al16(a.A) && al16(a.B) && al16(a.zeros) && a.K % 8 == 0 && a.lda % 8 == 0 &&
         a.ldb % 8 == 0 && (AK || a.M % 8 == 0) && (BK || a.N % 8 == 0);
}

template <typename T, typename TO, bool AK, bool BK, int EPI>
hipError_t launch(const GemmArgs& a, int splits, hipStream_t st) {
  if (a.seg_rows > 0) {
    // segmented B (the window weight gradients): the pipelined TN kernel on
    // 256 x 128 tiles, one workgroup per CU with a three-stage ring (measured
    // 8% faster than two 128 x 128 workgroups per CU with two stages each)
    if constexpr (sizeof(T) == 2 && !AK && !BK) {
      if (pipe_eligible<AK, BK>(a) && a.seg_rows % 64 == 0 && a.seg_count >= 1 && a.seg_first >= 0)
        return launch_pipe<TO, AK, BK, EPI, P256x128>(a, splits, st);
    }
    return hipErrorInvalidValue;
  }
  if constexpr (sizeof(T) == 2) {
    if (pipe_eligible<AK, BK>(a)) {
      switch (g_tile_override) {
        case 0: break;  // register-staged kernel, for comparison
        case 11: return launch_pipe<TO, AK, BK, EPI, P128x128>(a, splits, st);
        case 12: return launch_pipe<TO, AK, BK, EPI, P128x256>(a, splits, st);
        case 10: return launch_pipe<TO, AK, BK, EPI, P256x128>(a, splits, st);
        case 13: return launch_pipe<TO, AK, BK, EPI, P128x128o2>(a, splits, st);
        default:
          // The FFN up-projection and the input gradient through gelu'(u):
          // 256 x 256 tiles when they fill whole rounds of the CUs (measured
          // 13% and 2% faster per call at 8192 x 4096, 11% for the latter
          // with its per-panel aux loads). Otherwise weight gradients (both
          // operands MN-major) and the input gradient through gelu'(u): 128 x
          // 128 tiles, two workgroups per CU, so one's epilogue overlaps the
          // other's loop (3-6% faster for the latter, slower for the other
          // forward and input-gradient products); the rest: 256 x 128 tiles,
          // which re-read the weights half as often.
          if constexpr (AK && BK && (EPI == EPI_BIAS_GELU || EPI == EPI_GELU_GRAD)) {
            const int t256 = ((a.M + 255) / 256) * ((a.N + 255) / 256);
            if (splits == 1 && t256 % cu_count() == 0) return launch_pipe<TO, AK, BK, EPI, P256x256>(a, splits, st);
          }
          if constexpr (!AK || EPI == EPI_GELU_GRAD) return launch_pipe<TO, AK, BK, EPI, P128x128o2>(a, splits, st);
          else return launch_pipe<TO, AK, BK, EPI, P256x128>(a, splits, st);
      }
    }
  }
  hipError_t e = launch_cf<T, TO, AK, BK, EPI, T128x128>(a, splits, st);
  if constexpr (EPI != EPI_ATOMIC && EPI != EPI_ACC) {
    // the register-staged epilogue has no column sums: one pass over the output
    if (e == hipSuccess && a.colsum != nullptr)
      e = colsum_acc(sizeof(TO) == 2 ? DT_BF16 : DT_F32, a.C, a.ldc, a.M, a.N, a.colsum, st);
  }
  return e;
}

template <typename T, typename TO, bool AK, bool BK>
hipError_t by_epi(GemmEpi epi, const GemmArgs& a, int splits, hipStream_t st) {
  switch (epi) {
    case EPI_STORE: return launch<T, TO, AK, BK, EPI_STORE>(a, splits, st);
    case EPI_BIAS: return launch<T, TO, AK, BK, EPI_BIAS>(a, splits, st);
    case EPI_BIAS_RES: return launch<T, TO, AK, BK, EPI_BIAS_RES>(a, splits, st);
    case EPI_BIAS_GELU: return launch<T, TO, AK, BK, EPI_BIAS_GELU>(a, splits, st);
    case EPI_GELU_GRAD: return launch<T, TO, AK, BK, EPI_GELU_GRAD>(a, splits, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, bool AK, bool BK>
hipError_t by_epi_acc(GemmEpi epi, const GemmArgs& a, int splits, hipStream_t st) {
  if (epi == EPI_ACC) return launch<T, float, AK, BK, EPI_ACC>(a, 1, st);
  if (epi == EPI_ATOMIC) return launch<T, float, AK, BK, EPI_ATOMIC>(a, splits, st);
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t by_layout(bool out_f32, GemmLayout lay, GemmEpi epi, const GemmArgs& a, int splits, hipStream_t st) {
  if (epi == EPI_ACC || epi == EPI_ATOMIC) {
    // accumulation into fp32 is only used for weight gradients
    if (lay == GEMM_TN) return by_epi_acc<T, false, false>(epi, a, splits, st);
    return hipErrorInvalidValue;
  }
  if (splits != 1) return hipErrorInvalidValue;
  if (epi == EPI_CE_STATS || epi == EPI_CE_GRAD) {
    // pipelined bf16 kernel only; the statistics need 64-column groups
    if constexpr (sizeof(T) == 2) {
      if (lay != GEMM_NT || !pipe_eligible<true, true>(a) || a.row_tgt == nullptr || a.colsum != nullptr)
        return hipErrorInvalidValue;
      if (epi == EPI_CE_STATS) {
        if (a.ce_part == nullptr || a.ce_zt == nullptr || a.ld_part < (a.N + 63) / 64) return hipErrorInvalidValue;
        return launch_pipe<float, true, true, EPI_CE_STATS, P256x128>(a, 1, st);
      }
      if (a.row_lse == nullptr || out_f32) return hipErrorInvalidValue;
      return launch_pipe<T, true, true, EPI_CE_GRAD, P256x128>(a, 1, st);
    }
    return hipErrorInvalidValue;
  }
  if (lay == GEMM_NT) {
    if (out_f32) {
      if (epi != EPI_STORE) return hipErrorInvalidValue;
      return launch<T, float, true, true, EPI_STORE>(a, 1, st);
    }
    return by_epi<T, T, true, true>(epi, a, 1, st);
  }
  if (lay == GEMM_NN && !out_f32) {
    if (epi == EPI_STORE) return launch<T, T, true, false, EPI_STORE>(a, 1, st);
    if (epi == EPI_GELU_GRAD) return launch<T, T, true, false, EPI_GELU_GRAD>(a, 1, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace

void gemm_set_tile_override(int cfg) { g_tile_override = cfg; }

// Grouped weight gradients on 256 x 128 tiles (one workgroup per CU, three-stage
// ring) or 256 x 256 (two-stage ring), plain fp32 read-modify-write of each output tile.
namespace {
template <class CF> int group_tiles(int M, int N) { return ((M + CF::BM - 1) / CF::BM) * ((N + CF::BN - 1) / CF::BN); }
template <class CF> int group_xcd_m(int M, int N, int K) {
  const int tm = (M + CF::BM - 1) / CF::BM, tn = (N + CF::BN - 1) / CF::BN;
  int best = 0;
  double best_bytes = 0;
  for (int xm = 1; xm <= 8; xm *= 2) {
    const int xn = 8 / xm;
    if (tm % xm || tn % xn) continue;
    // panels one XCD reads: its bm row tiles of A and bn column tiles of B over K rows
    const double bytes = (double)K * 2.0 * ((tm / xm) * CF::BM + (tn / xn) * CF::BN);
    if (best == 0 || bytes < best_bytes) {
      best = xm;
      best_bytes = bytes;
    }
  }
  return best;
}
template <class CF, int EPI>
void launch_grouped(const GemmArgs& a, int total_tiles, int K, hipStream_t st) {
  hipLaunchKernelGGL((gemm_pipe_kernel<float, false, false, EPI, CF, true>), dim3(total_tiles, 1), dim3(CF::NT), 0, st,
                     a, K);
}
}  // namespace

int wgrad_group_tiles(int M, int N, bool wide) {
  return wide ? group_tiles<P256x256>(M, N) : group_tiles<P256x128>(M, N);
}

int wgrad_group_xcd_m(int M, int N, int K, bool wide) {
  return wide ? group_xcd_m<P256x256>(M, N, K) : group_xcd_m<P256x128>(M, N, K);
}

int wgrad_group_wide(const int* M, const int* N, int n) {
  const int cus = cu_count();
  auto padded = [](int t) { return (t + 7) / 8 * 8; };
  // cost in rounds of narrow tiles; n1 = 0 is the single narrow launch
  auto cost = [&](int n1) {
    int t1 = 0, t2 = 0;
    for (int p = 0; p < n; ++p) {
      if (p < n1) t1 += padded(group_tiles<P256x256>(M[p], N[p]));
      else t2 += padded(group_tiles<P256x128>(M[p], N[p]));
    }
    return 1.8 * ((t1 + cus - 1) / cus) + 1.0 * ((t2 + cus - 1) / cus);
  };
  int best = 0;
  double best_cost = cost(0);
  for (int n1 = n; n1 >= 1; --n1) {
    const double c = cost(n1);
    if (c < best_cost - 1e-9) {
      best = n1;
      best_cost = c;
    }
  }
  return best;
}

hipError_t gemm_wgrad_grouped(const WgradProblem* probs, int n, int total_tiles, int K, const void* zeros,
                              bool overwrite, bool wide, int* nonfinite, hipStream_t st) {
  if (probs == nullptr || n < 1 || total_tiles < 1 || K < 1 || K % 8 || zeros == nullptr ||
      (reinterpret_cast<uintptr_t>(zeros) & 15))
    return hipErrorInvalidValue;
  GemmArgs a{};
  a.K = K;
  a.zeros = zeros;
  a.group = probs;
  a.group_n = n;
  a.nonfinite = nonfinite;
  if (wide) {
    if (overwrite) launch_grouped<P256x256, EPI_STORE>(a, total_tiles, K, st);
    else launch_grouped<P256x256, EPI_ACC>(a, total_tiles, K, st);
  } else {
    if (overwrite) launch_grouped<P256x128, EPI_STORE>(a, total_tiles, K, st);
    else launch_grouped<P256x128, EPI_ACC>(a, total_tiles, K, st);
  }
  return hipGetLastError();
}

int gemm_acc_splits(DType dt, int M, int N, int K) {
  // Split-K count for Cf32 += A^T B. Cost model, in microseconds: rounds of
  // workgroups over the resident slots (CUs x workgroups per CU) times the
  // k-tiles each runs (about 2.3 TFLOP/s per CU, shared by its workgroups),
  // plus the fp32 read-modify-write or atomic adds of the epilogue (about
  // 2 ps per element and split).
  const bool pipe = dt == DT_BF16 && K % 8 == 0 && M % 8 == 0 && N % 8 == 0;
  const int bm = pipe ? P128x128o2::BM : T128x128::BM, bn = pipe ? P128x128o2::BN : T128x128::BN;
  const int bk = pipe ? 64 : KVN * (dt == DT_BF16 ? 8 : 4);
  const int occ = pipe ? P128x128o2::OCC : 1;   // workgroups resident per CU
  const int cus = cu_count() * occ;
  const double tiles = (double)((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  const int kt = (K + bk - 1) / bk;
  const double t_k = 2.0 * bm * bn * bk / (2.3e6 / occ), t_e = 2e-6 * M * N;
  int best = 1;
  double best_t = 1e30;
  for (int sp = 1; sp <= 16 && sp <= kt; sp *= 2) {
    const double rounds = std::ceil(tiles * sp / cus);
    const double t = rounds * std::ceil((double)kt / sp) * t_k + sp * t_e;
    if (t < best_t * 0.97) {
      best_t = t;
      best = sp;
    }
  }
  return best;
}

hipError_t gemm(DType dt, bool out_f32, GemmLayout lay, GemmEpi epi, const GemmArgs& a, int splits,
                hipStream_t st) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0 || splits < 1) return hipErrorInvalidValue;
  if (a.colsum != nullptr && (epi == EPI_ACC || epi == EPI_ATOMIC)) return hipErrorInvalidValue;
  if (dt == DT_BF16) return by_layout<bf16>(out_f32, lay, epi, a, splits, st);
  return by_layout<float>(out_f32, lay, epi, a, splits, st);
}

}  // namespace paci
