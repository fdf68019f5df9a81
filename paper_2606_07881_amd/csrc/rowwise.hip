// Bandwidth-bound row and column kernels: LayerNorm forward/backward and the
// column sums that feed bias and LayerNorm-affine gradients.
//
// LayerNorm uses one wavefront per row. The row is held in registers as
// 16-byte vectors (lane i owns vectors i, i + 64, ...), so each element is
// read once. Mean and variance are two-pass in fp32 with wavefront
// reductions. The affine gradients (sum of dn * xhat and of dn over rows) and
// the bias gradients are column reductions. A grid of (column slice, 64-row
// slice) workgroups streams the rows coalesced and adds its partial sums into
// the fp32 accumulator with atomics. The summation order is therefore free.
#include "device_common.hpp"
#include "kernels.hpp"

namespace paci {
namespace {

constexpr int NT = 256;

template <typename T> __device__ __forceinline__ u32x4 pack_vec(const float* f);
template <> __device__ __forceinline__ u32x4 pack_vec<float>(const float* f) {
  return u32x4{__builtin_bit_cast(uint32_t, f[0]), __builtin_bit_cast(uint32_t, f[1]),
               __builtin_bit_cast(uint32_t, f[2]), __builtin_bit_cast(uint32_t, f[3])};
}
template <> __device__ __forceinline__ u32x4 pack_vec<bf16>(const float* f) {
  return u32x4{pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]), pack_bf16x2(f[6], f[7])};
}

// ------------------------------------------------------------------------------------------
template <typename T, int MAXV>
__global__ void __launch_bounds__(NT) ln_fwd_kernel(const T* __restrict__ x, T* __restrict__ n, float* mean,
                                                     float* rstd, const float* __restrict__ gamma,
                                                     const float* __restrict__ beta, T* xcopy, int rows, int d,
                                                     float eps) {
  constexpr int V = Vec<T>::V;
  const int row = blockIdx.x * (NT / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int l = lane_id();
  const int nv = d / V;
  const T* xr = x + (int64_t)row * d;
  u32x4 xv[MAXV];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int vi = l + 64 * i;
    xv[i] = (vi < nv) ? ld16(xr + vi * V) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < V; ++j) s += vget<T>(xv[i], j);
  }
  const float mu = wave_sum(s) / d;
  float s2 = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    if (l + 64 * i < nv) {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const float c = vget<T>(xv[i], j) - mu;
        s2 += c * c;
      }
    }
  }
  const float rs = rsqrtf(wave_sum(s2) / d + eps);
  T* nr = n + (int64_t)row * d;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int vi = l + 64 * i;
    if (vi < nv) {
      float o[V];
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int c = vi * V + j;
        o[j] = (vget<T>(xv[i], j) - mu) * rs * gamma[c] + beta[c];
      }
      st16(nr + vi * V, pack_vec<T>(o));
      if (xcopy) st16(xcopy + (int64_t)row * d + vi * V, xv[i]);
    }
  }
  if (l == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

// ------------------------------------------------------------------------------------------
// dx for one row per wavefront (the affine gradients are a separate column pass).
template <typename T, int MAXV>
__global__ void __launch_bounds__(NT) ln_bwd_kernel(const T* __restrict__ dn, const T* __restrict__ x,
                                                     const float* __restrict__ mean, const float* __restrict__ rstd,
                                                     const float* __restrict__ gamma, const T* res, T* dx, int rows,
                                                     int d) {
  constexpr int V = Vec<T>::V;
  const int row = blockIdx.x * (NT / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int l = lane_id();
  const int nv = d / V;
  const float mu = mean[row], rs = rstd[row];
  const T* dnr = dn + (int64_t)row * d;
  const T* xr = x + (int64_t)row * d;
  u32x4 gv[MAXV], xv[MAXV];
  float sg = 0.f, sgx = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int vi = l + 64 * i;
    if (vi < nv) {
      gv[i] = ld16(dnr + vi * V);
      xv[i] = ld16(xr + vi * V);
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int c = vi * V + j;
        const float g = vget<T>(gv[i], j) * gamma[c];
        const float xh = (vget<T>(xv[i], j) - mu) * rs;
        sg += g;
        sgx += g * xh;
      }
    }
  }
  const float mg = wave_sum(sg) / d, mgx = wave_sum(sgx) / d;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int vi = l + 64 * i;
    if (vi < nv) {
      u32x4 rv = {0, 0, 0, 0};
      if (res) rv = ld16(res + (int64_t)row * d + vi * V);
      float o[V];
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int c = vi * V + j;
        const float xh = (vget<T>(xv[i], j) - mu) * rs;
        const float g = vget<T>(gv[i], j) * gamma[c];
        o[j] = rs * (g - mg - xh * mgx) + (res ? vget<T>(rv, j) : 0.f);
      }
      st16(dx + (int64_t)row * d + vi * V, pack_vec<T>(o));
    }
  }
}

// Column sums accumulated into fp32 with atomics. A workgroup of 256 threads
// is 8 row groups x 32 column vectors (16 bytes each). It covers
// 32 * V columns and CS_ROWS = 64 rows. Each thread issues its 8 row loads
// together, the 8 row groups are combined in LDS, and one thread per column
// adds the workgroup's sum into G. That is T / 64 atomic adds per column.
// With AFFINE, the sums are of dy * xhat and dy, where
// xhat = (x - mean) * rstd (the LayerNorm affine gradients), and, when G3 is
// given, of the rows of D as well (the LayerNorm's dx: the output-bias
// gradient of the linear layer before it).
constexpr int CS_THREADS = 256;
constexpr int CS_COLV = 32;             // column vectors per workgroup
constexpr int CS_RG = CS_THREADS / CS_COLV;
constexpr int CS_RPT = 8;               // rows per thread
constexpr int CS_ROWS = CS_RG * CS_RPT;
template <typename T, bool AFFINE>
__global__ void __launch_bounds__(CS_THREADS) colsum_atomic_kernel(const T* __restrict__ Y, int64_t ld, int rows,
                                                                    int ncols, const T* __restrict__ x,
                                                                    const float* __restrict__ mean,
                                                                    const float* __restrict__ rstd, float* G,
                                                                    float* G2, const T* __restrict__ D, float* G3) {
  constexpr int V = Vec<T>::V;
  __shared__ float red[AFFINE ? 3 : 1][CS_RG][CS_COLV * V];
  const int cv = threadIdx.x % CS_COLV, rg = threadIdx.x / CS_COLV;
  const int c0 = (blockIdx.x * CS_COLV + cv) * V;
  const bool colok = c0 < ncols;
  const int r0 = blockIdx.y * CS_ROWS + rg;
  const bool with_d = AFFINE && G3 != nullptr;   // uniform
  float a[V], b[V], e[V];
#pragma unroll
  for (int j = 0; j < V; ++j) a[j] = b[j] = e[j] = 0.f;
  u32x4 yv[CS_RPT], xv[CS_RPT], dv[CS_RPT];
#pragma unroll
  for (int i = 0; i < CS_RPT; ++i) {
    const int r = r0 + i * CS_RG;
    const bool ok = colok && r < rows;
    yv[i] = ok ? ld16(Y + (int64_t)r * ld + c0) : u32x4{0, 0, 0, 0};
    if (AFFINE) xv[i] = ok ? ld16(x + (int64_t)r * ld + c0) : u32x4{0, 0, 0, 0};
    if (AFFINE) dv[i] = (ok && with_d) ? ld16(D + (int64_t)r * ld + c0) : u32x4{0, 0, 0, 0};
  }
#pragma unroll
  for (int i = 0; i < CS_RPT; ++i) {
    const int r = r0 + i * CS_RG;
    if (AFFINE) {
      const bool ok = r < rows;
      const float mu = ok ? mean[r] : 0.f, rs = ok ? rstd[r] : 0.f;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const float g = vget<T>(yv[i], j);
        a[j] += g * (vget<T>(xv[i], j) - mu) * rs;
        b[j] += g;
        e[j] += vget<T>(dv[i], j);
      }
    } else {
#pragma unroll
      for (int j = 0; j < V; ++j) a[j] += vget<T>(yv[i], j);
    }
  }
#pragma unroll
  for (int j = 0; j < V; ++j) {
    red[0][rg][cv * V + j] = a[j];
    if (AFFINE) {
      red[AFFINE ? 1 : 0][rg][cv * V + j] = b[j];
      red[AFFINE ? 2 : 0][rg][cv * V + j] = e[j];
    }
  }
  __syncthreads();
  for (int c = threadIdx.x; c < CS_COLV * V; c += CS_THREADS) {
    const int col = blockIdx.x * CS_COLV * V + c;
    if (col >= ncols) continue;
    float sa = 0.f, sb = 0.f, se = 0.f;
#pragma unroll
    for (int g = 0; g < CS_RG; ++g) {
      sa += red[0][g][c];
      if (AFFINE) {
        sb += red[AFFINE ? 1 : 0][g][c];
        se += red[AFFINE ? 2 : 0][g][c];
      }
    }
    atomicAdd(G + col, sa);
    if (AFFINE) atomicAdd(G2 + col, sb);
    if (with_d) atomicAdd(G3 + col, se);
  }
}

template <typename T, int MAXV>
hipError_t ln_fwd_launch(const void* x, void* n, float* mean, float* rstd, const float* g, const float* b,
                         void* xcopy, int rows, int d, float eps, hipStream_t st) {
  hipLaunchKernelGGL((ln_fwd_kernel<T, MAXV>), dim3((rows + 3) / 4), dim3(NT), 0, st, reinterpret_cast<const T*>(x),
                     reinterpret_cast<T*>(n), mean, rstd, g, b, reinterpret_cast<T*>(xcopy), rows, d, eps);
  return hipGetLastError();
}

template <typename T, int MAXV>
hipError_t ln_bwd_launch(const void* dn, const void* x, const float* mean, const float* rstd, const float* gamma,
                         const void* res, void* dx, float* Gg, float* Gb, float* Gd, int rows, int d, hipStream_t st) {
  hipLaunchKernelGGL((ln_bwd_kernel<T, MAXV>), dim3((rows + 3) / 4), dim3(NT), 0, st, reinterpret_cast<const T*>(dn),
                     reinterpret_cast<const T*>(x), mean, rstd, gamma, reinterpret_cast<const T*>(res),
                     reinterpret_cast<T*>(dx), rows, d);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  constexpr int V = Vec<T>::V;
  const dim3 grid((d / V + CS_COLV - 1) / CS_COLV, (rows + CS_ROWS - 1) / CS_ROWS);
  hipLaunchKernelGGL((colsum_atomic_kernel<T, true>), grid, dim3(CS_THREADS), 0, st, reinterpret_cast<const T*>(dn),
                     (int64_t)d, rows, d, reinterpret_cast<const T*>(x), mean, rstd, Gg, Gb,
                     reinterpret_cast<const T*>(dx), Gd);
  return hipGetLastError();
}

template <typename T>
int maxv_for(int d) {
  const int nv = d / Vec<T>::V;
  return (nv + 63) / 64;
}

template <typename T>
hipError_t ln_fwd_t(const void* x, void* n, float* mean, float* rstd, const float* g, const float* b, void* xcopy,
                    int rows, int d, float eps, hipStream_t st) {
  const int mv = maxv_for<T>(d);
  if (mv <= 1) return ln_fwd_launch<T, 1>(x, n, mean, rstd, g, b, xcopy, rows, d, eps, st);
  if (mv <= 2) return ln_fwd_launch<T, 2>(x, n, mean, rstd, g, b, xcopy, rows, d, eps, st);
  if (mv <= 4) return ln_fwd_launch<T, 4>(x, n, mean, rstd, g, b, xcopy, rows, d, eps, st);
  if (mv <= 8) return ln_fwd_launch<T, 8>(x, n, mean, rstd, g, b, xcopy, rows, d, eps, st);
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t ln_bwd_t(const void* dn, const void* x, const float* mean, const float* rstd, const float* gamma,
                    const void* res, void* dx, float* Gg, float* Gb, float* Gd, int rows, int d, hipStream_t st) {
  const int mv = maxv_for<T>(d);
  if (mv <= 1) return ln_bwd_launch<T, 1>(dn, x, mean, rstd, gamma, res, dx, Gg, Gb, Gd, rows, d, st);
  if (mv <= 2) return ln_bwd_launch<T, 2>(dn, x, mean, rstd, gamma, res, dx, Gg, Gb, Gd, rows, d, st);
  if (mv <= 4) return ln_bwd_launch<T, 4>(dn, x, mean, rstd, gamma, res, dx, Gg, Gb, Gd, rows, d, st);
  if (mv <= 8) return ln_bwd_launch<T, 8>(dn, x, mean, rstd, gamma, res, dx, Gg, Gb, Gd, rows, d, st);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t layernorm_fwd(DType dt, const void* x, void* n, float* mean, float* rstd, const float* gamma,
                         const float* beta, void* xcopy, int rows, int d, float eps, hipStream_t st) {
  if (rows <= 0 || d <= 0 || d % 8) return hipErrorInvalidValue;
  if (dt == DT_BF16) return ln_fwd_t<bf16>(x, n, mean, rstd, gamma, beta, xcopy, rows, d, eps, st);
  return ln_fwd_t<float>(x, n, mean, rstd, gamma, beta, xcopy, rows, d, eps, st);
}

hipError_t layernorm_bwd(DType dt, const void* dn, const void* x, const float* mean, const float* rstd,
                         const float* gamma, const void* res, void* dx, float* Gg, float* Gb, float* Gd, int rows,
                         int d, hipStream_t st) {
  if (rows <= 0 || d <= 0 || d % 8) return hipErrorInvalidValue;
  if (dt == DT_BF16) return ln_bwd_t<bf16>(dn, x, mean, rstd, gamma, res, dx, Gg, Gb, Gd, rows, d, st);
  return ln_bwd_t<float>(dn, x, mean, rstd, gamma, res, dx, Gg, Gb, Gd, rows, d, st);
}

namespace {
// out = res + z * keep * scale, 8 consecutive elements per thread (one Philox
// draw). VEC: every pointer is 16-byte aligned, so the 8 elements move as
// 16-byte vectors (one for bf16, two for fp32).
template <typename T, bool VEC>
__global__ void __launch_bounds__(NT) dropout_kernel(const T* z, const T* res, T* out, int64_t n8, DropArgs drop) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (i >= n8) return;
  const uint64_t e8 = (uint64_t)i * 8;
  const uint32_t bits = drop_elem8(drop, e8);
  float zv[8], rv[8];
  if constexpr (VEC) {
    constexpr int NV = 8 * sizeof(T) / 16;   // 16-byte vectors per 8 elements
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const u32x4 a = ld16(z + e8 + q * (16 / sizeof(T)));
      const u32x4 b = res != nullptr ? ld16(res + e8 + q * (16 / sizeof(T))) : u32x4{0, 0, 0, 0};
#pragma unroll
      for (int j = 0; j < 16 / (int)sizeof(T); ++j) {
        zv[q * (16 / sizeof(T)) + j] = vget<T>(a, j);
        rv[q * (16 / sizeof(T)) + j] = vget<T>(b, j);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      zv[j] = to_f32(z[e8 + j]);
      rv[j] = res != nullptr ? to_f32(res[e8 + j]) : 0.f;
    }
  }
  float v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = (((bits >> j) & 1) ? zv[j] * drop.scale : 0.f) + rv[j];
  if constexpr (VEC && sizeof(T) == 2) {
    st16(out + e8, u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                         pack_bf16x2(v[6], v[7])});
  } else if constexpr (VEC) {
    st16(out + e8, __builtin_bit_cast(u32x4, floatx4{v[0], v[1], v[2], v[3]}));
    st16(out + e8 + 4, __builtin_bit_cast(u32x4, floatx4{v[4], v[5], v[6], v[7]}));
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) out[e8 + j] = from_f32<T>(v[j]);
  }
}

template <typename T>
void launch_dropout(const void* z, const void* res, void* out, int64_t n8, const DropArgs& drop, hipStream_t st) {
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  const dim3 grid((unsigned)((n8 + NT - 1) / NT));
  const T* zt = reinterpret_cast<const T*>(z);
  const T* rt = reinterpret_cast<const T*>(res);
  T* ot = reinterpret_cast<T*>(out);
  if (al16(z) && al16(out) && (res == nullptr || al16(res)))
    hipLaunchKernelGGL((dropout_kernel<T, true>), grid, dim3(NT), 0, st, zt, rt, ot, n8, drop);
  else
    hipLaunchKernelGGL((dropout_kernel<T, false>), grid, dim3(NT), 0, st, zt, rt, ot, n8, drop);
}
}  // namespace

hipError_t dropout_fwd(DType dt, const void* z, const void* res, void* out, int rows, int cols, const DropArgs& drop,
                       hipStream_t st) {
  if (rows <= 0 || cols <= 0 || cols % 8 || drop.thr == 0) return hipErrorInvalidValue;
  const int64_t n8 = (int64_t)rows * cols / 8;
  if (dt == DT_BF16) launch_dropout<bf16>(z, res, out, n8, drop, st);
  else launch_dropout<float>(z, res, out, n8, drop, st);
  return hipGetLastError();
}

hipError_t colsum_acc(DType dt, const void* Y, int64_t ld, int rows, int ncols, float* G, hipStream_t st) {
  if (rows <= 0 || ncols <= 0 || ncols % 8 || ld % 8) return hipErrorInvalidValue;
  const int V = (dt == DT_BF16) ? 8 : 4;
  const dim3 grid((ncols / V + CS_COLV - 1) / CS_COLV, (rows + CS_ROWS - 1) / CS_ROWS);
  if (dt == DT_BF16)
    hipLaunchKernelGGL((colsum_atomic_kernel<bf16, false>), grid, dim3(CS_THREADS), 0, st,
                       reinterpret_cast<const bf16*>(Y), ld, rows, ncols, nullptr, nullptr, nullptr, G, nullptr,
                       nullptr, nullptr);
  else
    hipLaunchKernelGGL((colsum_atomic_kernel<float, false>), grid, dim3(CS_THREADS), 0, st,
                       reinterpret_cast<const float*>(Y), ld, rows, ncols, nullptr, nullptr, nullptr, G, nullptr,
                       nullptr, nullptr);
  return hipGetLastError();
}

}  // namespace paci

// ============================================================================================
// First stage: embeddings. Last stage: softmax cross-entropy.
// ============================================================================================
namespace paci {
namespace {

template <typename T>
__global__ void __launch_bounds__(NT) embed_fwd_kernel(const int32_t* __restrict__ ids, const float* __restrict__ wte,
                                                        const float* __restrict__ wpe, T* x, int S, int d, int V,
                                                        int64_t total_vec) {
  const int64_t gv = (int64_t)blockIdx.x * NT + threadIdx.x;  // one vector of 4 columns
  if (gv >= total_vec) return;
  const int nv = d / 4;
  const int64_t t = gv / nv;
  const int c = (int)(gv % nv) * 4;
  const int s = (int)(t % S);
  const int id = ids[t];
  // ids outside [0, V) are a caller error; they read as a zero row instead of out of bounds
  const floatx4 a = (id >= 0 && id < V) ? *reinterpret_cast<const floatx4*>(wte + (int64_t)id * d + c)
                                        : floatx4{0.f, 0.f, 0.f, 0.f};
  const floatx4 b = *reinterpret_cast<const floatx4*>(wpe + (int64_t)s * d + c);
  T* o = x + t * d + c;
#pragma unroll
  for (int j = 0; j < 4; ++j) o[j] = from_f32<T>(a[j] + b[j]);
}

template <typename T>
__global__ void __launch_bounds__(NT) embed_bwd_wte_kernel(const int32_t* __restrict__ ids, const T* __restrict__ dx,
                                                            float* Gwte, int d, int V, int64_t total) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (i >= total) return;
  const int64_t t = i / d;
  const int c = (int)(i % d);
  const int id = ids[t];
  if (id < 0 || id >= V) return;
  atomicAdd(Gwte + (int64_t)id * d + c, to_f32(dx[i]));
}

template <typename T>
__global__ void __launch_bounds__(NT) embed_bwd_wpe_kernel(const T* __restrict__ dx, float* Gwpe, int mu, int S, int d) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;  // (s, c)
  if (i >= (int64_t)S * d) return;
  float acc = 0.f;
  for (int b = 0; b < mu; ++b) acc += to_f32(dx[(int64_t)b * S * d + i]);
  Gwpe[i] += acc;
}

__device__ __forceinline__ float block_reduce(float v, float* sh, bool is_max) {
  v = is_max ? wave_max(v) : wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if (lane_id() == 0) sh[w] = v;
  __syncthreads();
  float r = sh[0];
  for (int i = 1; i < NT / 64; ++i) r = is_max ? fmaxf(r, sh[i]) : r + sh[i];
  return r;
}

// One workgroup per token row.
__global__ void __launch_bounds__(NT) ce_fwd_kernel(const float* __restrict__ z, int64_t ldz,
                                                     const int32_t* __restrict__ tgt, float* lse, float* loss_row,
                                                     int V) {
  __shared__ float sh[NT / 64];
  const int64_t t = blockIdx.x;
  const float* zr = z + t * ldz;
  float mx = -INFINITY;
  for (int v = threadIdx.x; v < V; v += NT) mx = fmaxf(mx, zr[v]);
  mx = block_reduce(mx, sh, true);
  float s = 0.f;
  for (int v = threadIdx.x; v < V; v += NT) s += expf(zr[v] - mx);
  s = block_reduce(s, sh, false);
  if (threadIdx.x == 0) {
    const float l = mx + logf(s);
    const int y = tgt[t];
    lse[t] = l;
    // a target outside [0, V) is a caller error; it yields a NaN loss instead of an out-of-bounds read
    loss_row[t] = (y >= 0 && y < V) ? l - zr[y] : NAN;
  }
}

// Deterministic mean of T per-token losses: a single workgroup.
__global__ void __launch_bounds__(NT) mean_kernel(const float* __restrict__ x, int n, float* out) {
  __shared__ float sh[NT / 64];
  float s = 0.f;
  for (int i = threadIdx.x; i < n; i += NT) s += x[i];
  s = block_reduce(s, sh, false);
  if (threadIdx.x == 0) *out = s / n;
}

// One wavefront per token: lse from the (max, sum) partials of its 64-column
// groups, and its loss lse - z[target].
__global__ void __launch_bounds__(NT) ce_combine_kernel(const float2* __restrict__ part, int64_t ld_part,
                                                         int ngroups, const float* __restrict__ zt,
                                                         const int32_t* __restrict__ tgt, int V, float* lse,
                                                         float* loss_row, int T) {
  const int64_t t = (int64_t)blockIdx.x * (NT / 64) + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (t >= T) return;
  const float2* pr = part + t * ld_part;
  float mx = -INFINITY;
  for (int g = l; g < ngroups; g += 64) mx = fmaxf(mx, pr[g].x);
  mx = wave_max(mx);
  float s = 0.f;
  for (int g = l; g < ngroups; g += 64) {
    const float2 p = pr[g];
    s += p.y * expf(p.x - mx);
  }
  s = wave_sum(s);
  if (l == 0) {
    const float lt = mx + logf(s);
    const int y = tgt[t];
    lse[t] = lt;
    loss_row[t] = (y >= 0 && y < V) ? lt - zt[t] : NAN;
  }
}

template <typename T>
__global__ void __launch_bounds__(NT) ce_bwd_kernel(const float* __restrict__ z, int64_t ldz,
                                                     const int32_t* __restrict__ tgt, const float* __restrict__ lse,
                                                     T* dz, int V, float scale) {
  const int64_t t = blockIdx.x;
  const float* zr = z + t * ldz;
  T* dr = dz + t * ldz;
  const float l = lse[t];
  const int y = tgt[t];
  for (int v = threadIdx.x; v < ldz; v += NT) {
    float g = 0.f;
    if (v < V) g = scale * (expf(zr[v] - l) - (v == y ? 1.f : 0.f));
    dr[v] = from_f32<T>(g);
  }
}

}  // namespace

hipError_t embed_fwd(DType dt, const int32_t* ids, const float* wte, const float* wpe, void* x, int mu, int S, int d,
                     int V, hipStream_t st) {
  if (d % 4) return hipErrorInvalidValue;
  const int64_t total = (int64_t)mu * S * (d / 4);
  const dim3 grid((unsigned)((total + NT - 1) / NT));
  if (dt == DT_BF16)
    hipLaunchKernelGGL(embed_fwd_kernel<bf16>, grid, dim3(NT), 0, st, ids, wte, wpe, reinterpret_cast<bf16*>(x), S, d,
                       V, total);
  else
    hipLaunchKernelGGL(embed_fwd_kernel<float>, grid, dim3(NT), 0, st, ids, wte, wpe, reinterpret_cast<float*>(x), S,
                       d, V, total);
  return hipGetLastError();
}

hipError_t embed_bwd(DType dt, const int32_t* ids, const void* dx, float* Gwte, float* Gwpe, int mu, int S, int d,
                     int V, hipStream_t st) {
  const int64_t total = (int64_t)mu * S * d;
  const dim3 g1((unsigned)((total + NT - 1) / NT)), g2((unsigned)(((int64_t)S * d + NT - 1) / NT));
  if (dt == DT_BF16) {
    hipLaunchKernelGGL(embed_bwd_wte_kernel<bf16>, g1, dim3(NT), 0, st, ids, reinterpret_cast<const bf16*>(dx), Gwte,
                       d, V, total);
    hipLaunchKernelGGL(embed_bwd_wpe_kernel<bf16>, g2, dim3(NT), 0, st, reinterpret_cast<const bf16*>(dx), Gwpe, mu,
                       S, d);
  } else {
    hipLaunchKernelGGL(embed_bwd_wte_kernel<float>, g1, dim3(NT), 0, st, ids, reinterpret_cast<const float*>(dx), Gwte,
                       d, V, total);
    hipLaunchKernelGGL(embed_bwd_wpe_kernel<float>, g2, dim3(NT), 0, st, reinterpret_cast<const float*>(dx), Gwpe, mu,
                       S, d);
  }
  return hipGetLastError();
}

hipError_t ce_fwd(const float* z, int64_t ldz, const int32_t* tgt, float* lse, float* loss_out, float* part, int T,
                  int V, hipStream_t st) {
  hipLaunchKernelGGL(ce_fwd_kernel, dim3(T), dim3(NT), 0, st, z, ldz, tgt, lse, part, V);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(NT), 0, st, part, T, loss_out);
  return hipGetLastError();
}

int64_t ce_part_floats(int T) { return T; }

hipError_t ce_combine(const float* ce_part, int64_t ld_part, int ngroups, const float* zt, const int32_t* tgt, int V,
                      float* lse, float* loss_out, float* part_loss, int T, hipStream_t st) {
  if (T <= 0 || ngroups <= 0 || ld_part < ngroups || ngroups != (V + 63) / 64) return hipErrorInvalidValue;
  constexpr int RPB = NT / 64;
  hipLaunchKernelGGL(ce_combine_kernel, dim3((T + RPB - 1) / RPB), dim3(NT), 0, st,
                     reinterpret_cast<const float2*>(ce_part), ld_part, ngroups, zt, tgt, V, lse, part_loss, T);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(NT), 0, st, part_loss, T, loss_out);
  return hipGetLastError();
}

hipError_t ce_bwd(DType dt, const float* z, int64_t ldz, const int32_t* tgt, const float* lse, void* dz, int T, int V,
                  float scale, hipStream_t st) {
  if (dt == DT_BF16)
    hipLaunchKernelGGL(ce_bwd_kernel<bf16>, dim3(T), dim3(NT), 0, st, z, ldz, tgt, lse, reinterpret_cast<bf16*>(dz), V,
                       scale);
  else
    hipLaunchKernelGGL(ce_bwd_kernel<float>, dim3(T), dim3(NT), 0, st, z, ldz, tgt, lse, reinterpret_cast<float*>(dz),
                       V, scale);
  return hipGetLastError();
}

}  // namespace paci
