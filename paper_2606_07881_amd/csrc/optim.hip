// Fused AdamW over the flat parameter arena, and the fp32 -> bf16 refresh.
//
// One launch updates every parameter of the stage. Workgroup i takes entry i
// of a table built at init, each 4096 parameters of one tensor:
//   a range {begin, end, flags, 0} of a tensor, streamed as float4 vectors;
//   a 64 x 64 tile {offset, r0 << 16 | c0, flags | TILE, rows << 16 | cols} of a
//   block weight matrix [rows, cols]: the update as above, row by row, and the
//   tile's bf16 values transposed through LDS into the transposed working copy
//   [cols, rows] at the same offset, which the input-gradient products read.
// Per parameter: theta, G, m, v read (16 B); theta, m, v and the bf16 copy
// written (14 B), plus 2 B for the transposed copy of a block matrix and 4 B
// for G = 0 where the table asks for it (ranges whose G the next window's
// first backward does not overwrite).
#include <algorithm>

#include "device_common.hpp"
#include "kernels.hpp"

namespace paci {
namespace {

constexpr int NT = 256;

// Learning rate of update t (1-based): linear warmup, then a cosine down to
// lr_min_ratio of the peak at update lr_total; lr_total = 0: the constant rate.
__device__ double lr_at(const AdamwArgs& a, int t) {
  if (a.lr_total <= 0) return a.lr;
  if (t <= a.lr_warmup) return (double)a.lr * t / a.lr_warmup;
  const double p = fmin(1.0, (double)(t - a.lr_warmup) / (double)max(1, a.lr_total - a.lr_warmup));
  const double r = a.lr_min_ratio;
  return a.lr * (r + (1.0 - r) * 0.5 * (1.0 + cos(3.14159265358979323846 * p)));
}

__global__ void __launch_bounds__(NT) adamw_kernel(float* __restrict__ theta, float* __restrict__ G,
                                                    float* __restrict__ m, float* __restrict__ v,
                                                    bf16* __restrict__ theta16, bf16* __restrict__ theta16T,
                                                    const int4* __restrict__ chunks, AdamwArgs a,
                                                    const int* __restrict__ ctl) {
  __shared__ uint16_t tt[64][64 + 8];   // a tile's bf16 values, for the transposed copy
  const int4 ch = chunks[blockIdx.x];
  const bool tile = (ch.z & ADAMW_TILE) != 0, clear = (ch.z & ADAMW_CLEAR_G) != 0;
  const int rows = ch.w >> 16, cols = ch.w & 0xffff, r0 = ch.y >> 16, c0 = ch.y & 0xffff;
  const int rr = threadIdx.x >> 4, cc = (threadIdx.x & 15) * 4;   // tile: 16 rows of 16 float4 per pass
  auto st = [](float* p, floatx4 x) { __builtin_nontemporal_store(x, reinterpret_cast<floatx4*>(p)); };
  auto ld = [](const float* p) { return __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p)); };
  if (ctl[0] != 0) {   // non-finite G: no update; G cleared where the table asks
    if (!clear) return;
    if (tile) {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int r = r0 + 16 * p + rr, c = c0 + cc;
        if (r < rows && c < cols) st(G + ch.x + (int64_t)r * cols + c, floatx4{0.f, 0.f, 0.f, 0.f});
      }
    } else {
      for (int64_t i = (int64_t)ch.x + 4 * (int64_t)threadIdx.x; i < ch.y; i += 4 * NT)
        st(G + i, floatx4{0.f, 0.f, 0.f, 0.f});
    }
    return;
  }
  const int t = ctl[1] + 1;   // applied updates so far + 1: bias correction and schedule step
  const float lr = (float)lr_at(a, t);
  const float bc1 = (float)(1.0 - pow((double)a.beta1, (double)t));
  const float bc2 = (float)(1.0 - pow((double)a.beta2, (double)t));
  const float decay = (ch.z & ADAMW_DECAY) ? (1.f - lr * a.weight_decay) : 1.f;
  const float step = lr / bc1;
  const float rbc2 = 1.f / sqrtf(bc2);
  // every element is touched once: non-temporal loads and stores keep the
  // stream from displacing cached data
  auto math = [&](floatx4 g, floatx4& th, floatx4& mm, floatx4& vv) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      mm[j] = a.beta1 * mm[j] + (1.f - a.beta1) * g[j];
      vv[j] = a.beta2 * vv[j] + (1.f - a.beta2) * g[j] * g[j];
      const float denom = sqrtf(vv[j]) * rbc2 + a.eps;
      th[j] = th[j] * decay - step * mm[j] / denom;
    }
  };
  auto write = [&](int64_t i, floatx4 th, floatx4 mm, floatx4 vv) -> u32x2 {
    st(theta + i, th);
    st(m + i, mm);
    st(v + i, vv);
    if (clear) st(G + i, floatx4{0.f, 0.f, 0.f, 0.f});
    const u32x2 h = u32x2{pack_bf16x2(th[0], th[1]), pack_bf16x2(th[2], th[3])};
    if (theta16) __builtin_nontemporal_store(h, reinterpret_cast<u32x2*>(theta16 + i));
    return h;
  };
  if (tile) {
    // all loads of the tile first (16 float4 per thread in flight), then the math and stores
    floatx4 g[4], th[4], mm[4], vv[4];
    bool ok[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int r = r0 + 16 * p + rr, c = c0 + cc;
      ok[p] = r < rows && c < cols;
      const int64_t i = ch.x + (int64_t)r * cols + c;
      if (ok[p]) {
        g[p] = ld(G + i);
        th[p] = ld(theta + i);
        mm[p] = ld(m + i);
        vv[p] = ld(v + i);
      }
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      if (!ok[p]) continue;
      const int r = r0 + 16 * p + rr, c = c0 + cc;
      math(g[p], th[p], mm[p], vv[p]);
      const u32x2 h = write(ch.x + (int64_t)r * cols + c, th[p], mm[p], vv[p]);
      *reinterpret_cast<u32x2*>(&tt[16 * p + rr][cc]) = h;
    }
    if (theta16T == nullptr) return;   // uniform
    __syncthreads();
    // transposed copy [cols, rows]: row c0 + q / 8 gets 8 consecutive rows of the tile
#pragma unroll
    for (int q = threadIdx.x; q < 512; q += NT) {
      const int oc = q >> 3, part = q & 7;
      const int gr = c0 + oc, gc = r0 + part * 8;
      if (gr < cols && gc < rows) {
        u32x4 o;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          o[j] = (uint32_t)tt[part * 8 + 2 * j][oc] | ((uint32_t)tt[part * 8 + 2 * j + 1][oc] << 16);
        __builtin_nontemporal_store(o, reinterpret_cast<u32x4*>(theta16T + ch.x + (int64_t)gr * rows + gc));
      }
    }
    return;
  }
  // a range: two vectors per operand in flight per thread (the second one 4 NT elements on)
  int64_t i = (int64_t)ch.x + 4 * (int64_t)threadIdx.x;
  for (; i + 4 * NT < ch.y; i += 8 * NT) {
    const int64_t k = i + 4 * NT;
    const floatx4 g0 = ld(G + i), g1 = ld(G + k);
    floatx4 t0 = ld(theta + i), t1 = ld(theta + k);
    floatx4 m0 = ld(m + i), m1 = ld(m + k);
    floatx4 v0 = ld(v + i), v1 = ld(v + k);
    math(g0, t0, m0, v0);
    write(i, t0, m0, v0);
    math(g1, t1, m1, v1);
    write(k, t1, m1, v1);
  }
  if (i < ch.y) {
    const floatx4 g0 = ld(G + i);
    floatx4 t0 = ld(theta + i), m0 = ld(m + i), v0 = ld(v + i);
    math(g0, t0, m0, v0);
    write(i, t0, m0, v0);
  }
}

__global__ void __launch_bounds__(NT) fill_f32_kernel(float* __restrict__ p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < n; i += (int64_t)gridDim.x * NT) p[i] = v;
}

__global__ void __launch_bounds__(NT) f32_to_bf16_kernel(const float* __restrict__ src, bf16* dst, int64_t n) {
  const int64_t i = 4 * ((int64_t)blockIdx.x * NT + threadIdx.x);
  if (i + 3 < n) {
    const floatx4 x = *reinterpret_cast<const floatx4*>(src + i);
    *reinterpret_cast<u32x2*>(dst + i) = u32x2{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
  } else {
    for (int64_t j = i; j < n; ++j) dst[j] = (bf16)src[j];
  }
}

// ctl[0] = 1 if any element is NaN or infinite (ordinary vector stores; every
// writer stores the same value). Over all of G, or over the ranges of a table.
__global__ void __launch_bounds__(NT) guard_kernel(const floatx4* __restrict__ G, int64_t vecs, int* ctl) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < vecs; i += (int64_t)gridDim.x * NT) {
    const floatx4 g = G[i];
    bad |= !__builtin_isfinite(g[0]) | !__builtin_isfinite(g[1]) | !__builtin_isfinite(g[2]) |
           !__builtin_isfinite(g[3]);
  }
  if (bad) ctl[0] = 1;
}
__global__ void __launch_bounds__(NT) guard_ranges_kernel(const float* __restrict__ G, const int2* __restrict__ ranges,
                                                          int* ctl) {
  const int2 r = ranges[blockIdx.x];
  bool bad = false;
  for (int64_t i = (int64_t)r.x + 4 * (int64_t)threadIdx.x; i < r.y; i += 4 * NT) {
    const floatx4 g = *reinterpret_cast<const floatx4*>(G + i);
    bad |= !__builtin_isfinite(g[0]) | !__builtin_isfinite(g[1]) | !__builtin_isfinite(g[2]) |
           !__builtin_isfinite(g[3]);
  }
  if (bad) ctl[0] = 1;
}

// mode 0: clear the non-finite flag; 1: count the update as applied or skipped
// and clear the flag for the next window; 2: clear every counter.
__global__ void ctl_kernel(int* ctl, int mode) {
  if (threadIdx.x != 0) return;
  if (mode == 0) {
    ctl[0] = 0;
  } else if (mode == 1) {
    if (ctl[0]) ctl[2] = ctl[2] + 1;
    else ctl[1] = ctl[1] + 1;
    ctl[0] = 0;
  } else {
    ctl[0] = ctl[1] = ctl[2] = ctl[3] = 0;
  }
}

// dst [cols, rows] = src [rows, cols]^T, 16-bit elements, through a 64 x 64 LDS
// tile; rows and cols multiples of 8 (whole 16-byte vectors on both sides).
__global__ void __launch_bounds__(NT) transpose16_kernel(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                                                         int rows, int cols) {
  __shared__ uint16_t t[64][64 + 8];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  for (int q = threadIdx.x; q < 512; q += NT) {
    const int r = q >> 3, ch = q & 7;
    const int gr = r0 + r, gc = c0 + ch * 8;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (gr < rows && gc < cols) v = *reinterpret_cast<const u32x4*>(src + (int64_t)gr * cols + gc);
    *reinterpret_cast<u32x4*>(&t[r][ch * 8]) = v;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < 512; q += NT) {
    const int cc = q >> 3, ch = q & 7;
    const int gr = c0 + cc, gc = r0 + ch * 8;
    if (gr < cols && gc < rows) {
      u32x4 o;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        o[j] = (uint32_t)t[ch * 8 + 2 * j][cc] | ((uint32_t)t[ch * 8 + 2 * j + 1][cc] << 16);
      *reinterpret_cast<u32x4*>(dst + (int64_t)gr * rows + gc) = o;
    }
  }
}

}  // namespace

hipError_t transpose16(const void* src, void* dst, int rows, int cols, hipStream_t st) {
  if (rows <= 0 || cols <= 0 || rows % 8 || cols % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(transpose16_kernel, dim3((cols + 63) / 64, (rows + 63) / 64), dim3(NT), 0, st,
                     reinterpret_cast<const uint16_t*>(src), reinterpret_cast<uint16_t*>(dst), rows, cols);
  return hipGetLastError();
}

hipError_t adamw(float* theta, float* G, float* m, float* v, void* theta_bf16, void* theta_bf16T, const int4* chunks,
                 int nchunks, const AdamwArgs& a, const int* ctl, hipStream_t st) {
  if (nchunks <= 0 || ctl == nullptr) return hipErrorInvalidValue;
  hipLaunchKernelGGL(adamw_kernel, dim3(nchunks), dim3(NT), 0, st, theta, G, m, v, reinterpret_cast<bf16*>(theta_bf16),
                     reinterpret_cast<bf16*>(theta_bf16T), chunks, a, ctl);
  return hipGetLastError();
}

hipError_t adamw_guard_ranges(const float* G, const int2* ranges, int nranges, int* ctl, hipStream_t st) {
  if (nranges < 0 || ctl == nullptr) return hipErrorInvalidValue;
  if (nranges == 0) return hipSuccess;
  hipLaunchKernelGGL(guard_ranges_kernel, dim3(nranges), dim3(NT), 0, st, G, ranges, ctl);
  return hipGetLastError();
}

hipError_t adamw_guard(const float* G, int64_t n, int* ctl, hipStream_t st) {
  if (n <= 0 || n % 4) return hipErrorInvalidValue;
  const int64_t vecs = n / 4;
  const int blocks = (int)std::min<int64_t>(4096, (vecs + NT - 1) / NT);
  hipLaunchKernelGGL(guard_kernel, dim3(blocks), dim3(NT), 0, st, reinterpret_cast<const floatx4*>(G), vecs, ctl);
  return hipGetLastError();
}

hipError_t adamw_ctl(int* ctl, int mode, hipStream_t st) {
  if (mode < 0 || mode > 2) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ctl_kernel, dim3(1), dim3(64), 0, st, ctl, mode);
  return hipGetLastError();
}

hipError_t fill_f32(float* p, int64_t n, float v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>(2048, (n + NT - 1) / NT);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(blocks), dim3(NT), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t f32_to_bf16(const float* src, void* dst, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 4 * NT - 1) / (4 * NT);
  hipLaunchKernelGGL(f32_to_bf16_kernel, dim3((unsigned)blocks), dim3(NT), 0, st, src, reinterpret_cast<bf16*>(dst), n);
  return hipGetLastError();
}

}  // namespace paci
