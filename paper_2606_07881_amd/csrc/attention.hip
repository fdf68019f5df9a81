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
#include "device_common.hpp"
#include "kernels.hpp"

namespace paci {
namespace {

constexpr int NT = 256;
constexpr int BKV = 64;   // keys per block
constexpr float LOG2E = 1.4426950408889634f;

// ---------------------------------------------------------------------------------------
template <typename T, int DH>
__global__ void __launch_bounds__(NT) attn_fwd_kernel(const T* qkv, T* out, float* lse2, int S, int H, int d,
                                                       float scale_log2) {
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
template <typename T, int DH>
__global__ void __launch_bounds__(NT) attn_bwd_dkdv_kernel(const T* qkv, const T* dO, const float* lse2,
                                                            const float* Dsum, T* dqkv, int S, int H, int d,
                                                            float scale_log2, float scale) {
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
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qi = qt * 16 + 4 * (l >> 4) + r;
        const int q = q0 + qi;
        const bool ok = (key <= q) && (q < S) && (key < S);
        const float p = ok ? exp2f(s[r] * scale_log2 - sL[qi]) : 0.f;
        P[qt][r] = p;
        dS[qt][r] = p * (dp[r] - sD[qi]);
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

template <typename T, int DH>
__global__ void __launch_bounds__(NT) attn_bwd_dq_kernel(const T* qkv, const T* dO, const float* lse2,
                                                          const float* Dsum, T* dqkv, int S, int H, int d,
                                                          float scale_log2, float scale) {
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
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + kt * 16 + 4 * (l >> 4) + r;
        const bool ok = qok && (key <= qrow) && (key < S);
        const float p = ok ? exp2f(s[r] * scale_log2 - lq) : 0.f;
        dS[kt][r] = p * (dp[r] - Dq);
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

template <typename T, int DH>
hipError_t fwd_launch(const void* qkv, void* o, float* lse2, int mu, int S, int H, hipStream_t st) {
  const int d = H * DH;
  const float scale_log2 = LOG2E / sqrtf((float)DH);
  dim3 grid((S + 63) / 64, mu * H);
  hipLaunchKernelGGL((attn_fwd_kernel<T, DH>), grid, dim3(NT), 0, st, reinterpret_cast<const T*>(qkv),
                     reinterpret_cast<T*>(o), lse2, S, H, d, scale_log2);
  return hipGetLastError();
}

template <typename T, int DH>
hipError_t bwd_launch(const void* qkv, const void* o, const void* dO, const float* lse2, float* Dbuf, void* dqkv,
                      int mu, int S, int H, hipStream_t st) {
  const int d = H * DH;
  const float scale = 1.f / sqrtf((float)DH);
  const float scale_log2 = LOG2E * scale;
  constexpr int LPR = DH / Vec<T>::V;
  const int64_t rows = (int64_t)mu * S * H;
  const int64_t threads = rows * LPR;
  hipLaunchKernelGGL((attn_dsum_kernel<T, DH>), dim3((unsigned)((threads + NT - 1) / NT)), dim3(NT), 0, st,
                     reinterpret_cast<const T*>(o), reinterpret_cast<const T*>(dO), Dbuf, S, H, d, rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, DH>), dim3((S + BKV - 1) / BKV, mu * H), dim3(NT), 0, st,
                     reinterpret_cast<const T*>(qkv), reinterpret_cast<const T*>(dO), lse2, Dbuf,
                     reinterpret_cast<T*>(dqkv), S, H, d, scale_log2, scale);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<T, DH>), dim3((S + 63) / 64, mu * H), dim3(NT), 0, st,
                     reinterpret_cast<const T*>(qkv), reinterpret_cast<const T*>(dO), lse2, Dbuf,
                     reinterpret_cast<T*>(dqkv), S, H, d, scale_log2, scale);
  return hipGetLastError();
}

template <typename T>
hipError_t fwd_dh(const void* qkv, void* o, float* lse2, int mu, int S, int H, int dh, hipStream_t st) {
  switch (dh) {
    case 32: return fwd_launch<T, 32>(qkv, o, lse2, mu, S, H, st);
    case 64: return fwd_launch<T, 64>(qkv, o, lse2, mu, S, H, st);
    case 128:
      // fp32 at head_dim 128 would exceed the 64 KiB LDS budget of these tilings
      if constexpr (sizeof(T) == 2) return fwd_launch<T, 128>(qkv, o, lse2, mu, S, H, st);
      break;
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t bwd_dh(const void* qkv, const void* o, const void* dO, const float* lse2, float* Dbuf, void* dqkv,
                  int mu, int S, int H, int dh, hipStream_t st) {
  switch (dh) {
    case 32: return bwd_launch<T, 32>(qkv, o, dO, lse2, Dbuf, dqkv, mu, S, H, st);
    case 64: return bwd_launch<T, 64>(qkv, o, dO, lse2, Dbuf, dqkv, mu, S, H, st);
    case 128:
      if constexpr (sizeof(T) == 2) return bwd_launch<T, 128>(qkv, o, dO, lse2, Dbuf, dqkv, mu, S, H, st);
      break;
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t attn_fwd(DType dt, const void* qkv, void* o, float* lse2, int mu, int S, int H, int dh, hipStream_t st) {
  if (mu <= 0 || S <= 0 || H <= 0) return hipErrorInvalidValue;
  if (dt == DT_BF16) return fwd_dh<bf16>(qkv, o, lse2, mu, S, H, dh, st);
  return fwd_dh<float>(qkv, o, lse2, mu, S, H, dh, st);
}

hipError_t attn_bwd(DType dt, const void* qkv, const void* o, const void* dO, const float* lse2, float* Dbuf,
                    void* dqkv, int mu, int S, int H, int dh, hipStream_t st) {
  if (mu <= 0 || S <= 0 || H <= 0) return hipErrorInvalidValue;
  if (dt == DT_BF16) return bwd_dh<bf16>(qkv, o, dO, lse2, Dbuf, dqkv, mu, S, H, dh, st);
  return bwd_dh<float>(qkv, o, dO, lse2, Dbuf, dqkv, mu, S, H, dh, st);
}

}  // namespace paci
