// Matrix-core GEMM for the stage's linear layers (forward, input gradient and
// weight gradient with fused fp32 accumulation), gfx950.
//
// Work decomposition: one 256-thread workgroup (4 wavefronts, 2 x 2) per
// 128 x 128 output tile; each wavefront owns a 64 x 64 sub-tile = 4 x 4 MFMA
// 16 x 16 tiles. The contracted dimension advances in 8-vector slices (64 bf16 or
// 32 fp32 elements), double-buffered in LDS: the global loads of slice k+1 are
// in flight while slice k is multiplied. Operands stored contracted-major
// (K-major) are copied as 16-byte vectors. Operands stored the other way
// (MN-major: the weight in dX = dY W, both activations in dW = dY^T X) are
// loaded as V x V blocks and transposed in registers before the LDS write, so
// every LDS fragment read is one 16-byte access.
//
// Tile order is XCD-aware: workgroup w runs on XCD w % 8, so each XCD gets a
// contiguous range of tiles, walked in groups of 8 tile-rows to keep A and B
// panels in that XCD's L2.
#include "device_common.hpp"
#include "kernels.hpp"

namespace paci {
namespace {

constexpr int BM = 128, BN = 128, WM = 64, WN = 64, NT = 256, KVN = 8, GROUP_M = 8;

// Register-staged tile loader (global -> registers -> LDS).
template <typename T, int ROWS, bool KMAJ>
struct TileLoader {
  static constexpr int V = Vec<T>::V;
  static constexpr int ITEMS = KMAJ ? ROWS * KVN : (ROWS / V) * KVN;
  static constexpr int PT = (ITEMS + NT - 1) / NT;
  static constexpr int NV = KMAJ ? 1 : V;
  u32x4 r[PT][NV];

  // rows [row0, row0+ROWS) of `rows_total`; contracted [k0, k0 + 8V) of k_end.
  __device__ __forceinline__ void load(const T* src, int64_t ld, int row0, int rows_total, int k0, int k_end,
                                       int tid) {
#pragma unroll
    for (int p = 0; p < PT; ++p) {
      const int it = tid + p * NT;
      if ((ITEMS % NT) != 0 && it >= ITEMS) continue;
      const int kv = it % KVN, rr = it / KVN;
      if (KMAJ) {
        const int row = row0 + rr, k = k0 + kv * V;
        u32x4 v = {0, 0, 0, 0};
        if (row < rows_total && k < k_end) {
          v = ld16(src + (int64_t)row * ld + k);
          if (k + V > k_end) v = vmask_tail<T>(v, k_end - k);
        }
        r[p][0] = v;
      } else {
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
      const int kv = it % KVN, rr = it / KVN;
      if (KMAJ) {
        tile[lds_slot<ROWS>(kv, rr)] = r[p][0];
      } else {
        u32x4 out[V];
        transpose_block<T>(r[p], out);
#pragma unroll
        for (int i = 0; i < V; ++i) tile[lds_slot<ROWS>(kv, rr * V + i)] = out[i];
      }
    }
  }
};

__device__ __forceinline__ float gelu_f(float u) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  return 0.5f * u * (1.0f + tanhf(c * (u + a * u * u * u)));
}
__device__ __forceinline__ float gelu_grad_f(float u) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  const float th = tanhf(c * (u + a * u * u * u));
  return 0.5f * (1.0f + th) + 0.5f * u * (1.0f - th * th) * c * (1.0f + 3.0f * a * u * u);
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
  float o[4];
  for (int j = 0; j < 4; ++j) {
    float x = acc[j];
    const int nn = n + (j < nv ? j : 0);
    if (EPI == EPI_BIAS || EPI == EPI_BIAS_RES || EPI == EPI_BIAS_GELU) x += a.bias[nn];
    if (EPI == EPI_BIAS_RES) x += ldf<T>(a.aux, (int64_t)m * a.ld_aux + nn);
    if (EPI == EPI_GELU_GRAD) x *= gelu_grad_f(ldf<T>(a.aux, (int64_t)m * a.ld_aux + nn));
    o[j] = x;
  }
  store4<TO>(reinterpret_cast<TO*>(a.C), (int64_t)m * a.ldc + n, o, nv);
  if (EPI == EPI_BIAS_GELU) {
    for (int j = 0; j < 4; ++j) o[j] = gelu_f(o[j]);
    store4<TO>(reinterpret_cast<TO*>(a.C2), (int64_t)m * a.ldc + n, o, nv);
  }
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

template <typename T, typename TO, bool AK, bool BK, int EPI>
__global__ void __launch_bounds__(NT, 2) gemm_kernel(GemmArgs a, int k_per_split) {
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
  const int wm0 = (w >> 1) * WM, wn0 = (w & 1) * WN;

  const T* A = reinterpret_cast<const T*>(a.A);
  const T* B = reinterpret_cast<const T*>(a.B);
  TileLoader<T, BM, AK> la;
  TileLoader<T, BN, BK> lb;
  // When both operands are MN-major each uses half of the threads.
  const int tid_b = (!AK && !BK) ? ((tid + NT / 2) % NT) : tid;

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
      for (int i = 0; i < WM / 16; ++i) yf[i] = lds_frag<BM>(sa, s, wm0 + i * 16);
#pragma unroll
      for (int j = 0; j < WN / 16; ++j) xf[j] = lds_frag<BN>(sb, s, wn0 + j * 16);
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

template <typename T, typename TO, bool AK, bool BK, int EPI>
hipError_t launch(const GemmArgs& a, int splits, hipStream_t st) {
  constexpr int BKE = KVN * Vec<T>::V;
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  int kps = (a.K + splits - 1) / splits;
  kps = ((kps + BKE - 1) / BKE) * BKE;
  const int used = (a.K + kps - 1) / kps;
  hipLaunchKernelGGL((gemm_kernel<T, TO, AK, BK, EPI>), dim3(tiles, used), dim3(NT), 0, st, a, kps);
  return hipGetLastError();
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

int gemm_tile_m() { return BM; }
int gemm_tile_n() { return BN; }
int gemm_tile_k(DType dt) { return KVN * (dt == DT_BF16 ? 8 : 4); }

hipError_t gemm(DType dt, bool out_f32, GemmLayout lay, GemmEpi epi, const GemmArgs& a, int splits,
                hipStream_t st) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0 || splits < 1) return hipErrorInvalidValue;
  if (dt == DT_BF16) return by_layout<bf16>(out_f32, lay, epi, a, splits, st);
  return by_layout<float>(out_f32, lay, epi, a, splits, st);
}

}  // namespace paci
