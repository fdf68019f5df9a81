// Device-side building blocks shared by the stage kernels (gfx950 / CDNA4).
//
// Matrix-core convention used everywhere
// --------------------------------------
// One MFMA "step" contracts 4 * V elements, where V = 16 bytes / sizeof(T)
// (8 for bf16, 4 for fp32). In a step, lane l of a 64-wide wavefront supplies
// one 16-byte vector per operand: row (l % 16) of a 16-row operand tile, and
// the V contracted elements of group g = l / 16. bf16 uses one
// v_mfma_f32_16x16x32_bf16 per step. fp32 uses four v_mfma_f32_16x16x4_f32,
// the j-th taking element j of each lane's vector. Both operands use the same
// lane -> contracted-index assignment, so any consistent permutation of the
// contracted index inside a step gives the same sum.
//
// mma_step(acc, X, Y) accumulates D += X Y^T for two 16-row tiles X and Y. Lane
// l then holds D[4 * (l / 16) + r][l % 16], r = 0..3: four consecutive X-rows
// of one Y-row.
//
// LDS tile layout: a tile of R rows by 8 vectors (8 * V contracted elements)
// is stored as [kv][row], one 16-byte slot each. The row is XOR-swizzled with
// the vector index (physical row = row ^ (kv & 7)). This keeps conflict-free
// 16-byte accesses for the three patterns the kernels use: 8 lanes writing
// one row's 8 vectors, 8 lanes writing 8 vectors of a transposed 8x8 block,
// and 16 lanes reading 16 consecutive rows of one vector index.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace paci {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float floatx4 __attribute__((__vector_size__(4 * sizeof(float))));
typedef uint32_t u32x4 __attribute__((__vector_size__(4 * sizeof(uint32_t))));
typedef uint32_t u32x2 __attribute__((__vector_size__(2 * sizeof(uint32_t))));

template <typename T> struct Vec { static constexpr int V = 16 / sizeof(T); };

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// ---- element access inside a raw 16-byte vector -----------------------------------
// Reinterpret one 32-bit word. The word is taken by value: applying
// __builtin_bit_cast directly to an element of a vector reference (v[j]) was
// compiled as a read of element 0 for every j by this toolchain.
__device__ __forceinline__ float as_float(uint32_t w) { return __builtin_bit_cast(float, w); }

template <typename T> __device__ __forceinline__ float vget(const u32x4& v, int j);
template <> __device__ __forceinline__ float vget<float>(const u32x4& v, int j) {
  const uint32_t w = v[j];
  return as_float(w);
}
template <> __device__ __forceinline__ float vget<bf16>(const u32x4& v, int j) {
  uint32_t w = v[j >> 1];
  return __builtin_bit_cast(float, (j & 1) ? (w & 0xffff0000u) : (w << 16));
}

// Zero the elements j >= n of a vector (n in [0, V]).
template <typename T> __device__ __forceinline__ u32x4 vmask_tail(u32x4 v, int n) {
  constexpr int V = Vec<T>::V;
  if (n >= V) return v;
  if (sizeof(T) == 4) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j >= n) v[j] = 0;
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (2 * w >= n) v[w] = 0;
      else if (2 * w + 1 >= n) v[w] &= 0xffffu;
    }
  }
  return v;
}

// Transpose a V x V block held as V row vectors: out[i] gathers element i of
// every input row, in row order.
template <typename T> __device__ __forceinline__ void transpose_block(const u32x4* in, u32x4* out);
template <> __device__ __forceinline__ void transpose_block<float>(const u32x4* in, u32x4* out) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) out[i][j] = in[j][i];
}
template <> __device__ __forceinline__ void transpose_block<bf16>(const u32x4* in, u32x4* out) {
  // out[i] word p = (element i of row 2p) | (element i of row 2p+1) << 16
#pragma unroll
  for (int i = 0; i < 8; ++i) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t a = in[2 * p][i >> 1], b = in[2 * p + 1][i >> 1];
      out[i][p] = (i & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
  }
}

// ---- MFMA step ---------------------------------------------------------------------
template <typename T> __device__ __forceinline__ void mma_step(floatx4& acc, const u32x4& x, const u32x4& y);
template <> __device__ __forceinline__ void mma_step<bf16>(floatx4& acc, const u32x4& x, const u32x4& y) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, x), __builtin_bit_cast(bf16x8, y),
                                                acc, 0, 0, 0);
}
template <> __device__ __forceinline__ void mma_step<float>(floatx4& acc, const u32x4& x, const u32x4& y) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
  {
    const uint32_t xw = x[j], yw = y[j];
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(as_float(xw), as_float(yw), acc, 0, 0, 0);
  }
}

// ---- swizzled LDS tile addressing ------------------------------------------------------
template <int ROWS> __device__ __forceinline__ int lds_slot(int kv, int row) {
  return kv * ROWS + (row ^ (kv & 7));
}

// Fragment of a 16-row operand tile for MFMA step `s` (rows row0 .. row0+15).
template <int ROWS> __device__ __forceinline__ u32x4 lds_frag(const u32x4* tile, int s, int row0) {
  const int l = lane_id();
  const int kv = s * 4 + (l >> 4);
  return tile[lds_slot<ROWS>(kv, row0 + (l & 15))];
}

// ---- MN-major bf16 tiles read with the LDS transpose instruction ----------------------
// A bf16 operand stored with its rows (m or n) contiguous and the contracted
// index k as the outer dimension is staged in LDS as [k][ROWS] (16-byte
// chunks of 8 rows), with chunk c of line k stored at chunk c ^ ((k & 3) << 1).
// ds_read_b64_tr_b16 gives each lane j of a 16-lane group 4 values
// (element i from the 8 bytes addressed by lane 4i + j / 4, position j % 4).
// If lane c addresses line kb + c / 4, rows r0 + 4 (c % 4) .. + 3, lane j
// receives rows r0 + j of lines kb .. kb + 3. Two such reads (kb and kb + 4)
// give the 8 contracted values an MFMA step wants, with no register transpose.
// MN-major operand tile in LDS: row k holds ROWS elements as 16-byte chunks,
// chunk j stored at chunk j ^ trt_swz(k). A transpose read takes 4 rows x 2
// chunks per 16 lanes, and the hardware serves two such lane groups (rows k
// and k + 8) per cycle: bits 1-2 of the swizzle separate the 4 rows of a
// group, bit 3 the two groups, so the 64 banks are hit once per cycle.
template <int ROWS> __device__ __forceinline__ int trt_swz(int k) {
  if constexpr (ROWS >= 128) return ((k & 3) << 1) ^ (((k >> 3) & 1) << 3);
  else return (k & 3) << 1;
}
template <int ROWS> __device__ __forceinline__ int trt_elem(int k, int r) {
  return k * ROWS + (((r >> 3) ^ trt_swz<ROWS>(k)) << 3) + (r & 7);
}
typedef short i16x4 __attribute__((ext_vector_type(4)));
// The same read from a precomputed address: off = lds_frag_tr_off<ROWS>(row0)
// is this lane's byte offset within the tile for step 0, and the tile's LDS
// byte address is added per read. Lines k0 + 4 and k0 + 32 s keep the swizzle
// of line k0 (k0 = 8 g + 0..3 leaves bits 0, 1 and 3 unchanged by those
// steps), so both reads of any step are constant offsets from it.
template <int ROWS> __device__ __forceinline__ uint32_t lds_frag_tr_off(int row0) {
  const int l = lane_id();
  const int g = l >> 4, c = l & 15;
  return (uint32_t)(2 * trt_elem<ROWS>(8 * g + (c >> 2), row0 + 4 * (c & 3)));
}
template <int ROWS> __device__ __forceinline__ u32x4 lds_frag_tr_at(uint32_t addr, int s) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const uint32_t a0 = addr + (uint32_t)(s * 32 * ROWS * 2);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(uintptr_t)a0);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(uintptr_t)(a0 + 4 * ROWS * 2));
  const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  return u32x4{a[0], a[1], b[0], b[1]};
}
template <int ROWS> __device__ __forceinline__ u32x4 lds_frag_tr(const u32x4* tile, int s, int row0) {
  const int l = lane_id();
  const int g = l >> 4, c = l & 15;
  const bf16* base = reinterpret_cast<const bf16*>(tile);
  const int r = row0 + 4 * (c & 3);
  const int k0 = s * 32 + 8 * g + (c >> 2);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(base + trt_elem<ROWS>(k0, r)));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(base + trt_elem<ROWS>(k0 + 4, r)));
  const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  return u32x4{a[0], a[1], b[0], b[1]};
}

// ---- wave reductions ---------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
// Reduce across the four 16-lane groups (lanes l, l^16, l^32, l^48).
__device__ __forceinline__ float group4_sum(float v) {
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}
__device__ __forceinline__ float group4_max(float v) {
  v = fmaxf(v, __shfl_xor(v, 16, 64));
  v = fmaxf(v, __shfl_xor(v, 32, 64));
  return v;
}

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }
// The same through global-address-space pointers, for data known to be in
// device memory: global_* instructions count in vmcnt only, where flat_* ones
// (the compiler's choice for a pointer it cannot place) also count in
// lgkmcnt and so hold up every later wait for LDS reads.
__device__ __forceinline__ u32x4 ld16g(const void* p) {
  return *(const __attribute__((address_space(1))) u32x4*)p;
}
__device__ __forceinline__ void st16g(void* p, const u32x4& v) { *(__attribute__((address_space(1))) u32x4*)p = v; }

// ---- one-shot tile staging (global -> LDS), used by the attention kernels -----------------
// K-major source: element (row r, contracted c) at src[r * ld + c]. Stages rows
// [0, ROWS) and contracted vectors [0, KVN); rows >= rows_valid read as zero.
template <typename T, int ROWS, int KVN, int NT>
__device__ __forceinline__ void stage_kmajor(u32x4* tile, const T* src, int ld, int rows_valid) {
  constexpr int V = Vec<T>::V;
  constexpr int ITEMS = ROWS * KVN;
#pragma unroll
  for (int it = threadIdx.x; it < ITEMS; it += NT) {
    const int kv = it % KVN, r = it / KVN;
    u32x4 v = {0, 0, 0, 0};
    if (r < rows_valid) v = ld16(src + (size_t)r * ld + kv * V);
    tile[lds_slot<ROWS>(kv, r)] = v;
  }
}

// MN-major source: element (contracted c, row r) at src[c * ld + r]. The
// contracted index of element j of vector kv is perm(kv, j) (a permutation of
// 0 .. KVN*V-1 that keeps each MFMA step's 4*V indices together). Contracted
// indices >= c_valid read as zero. Rows [0, ROWS) must be in bounds.
template <typename T, int ROWS, int KVN, int NT, class Perm>
__device__ __forceinline__ void stage_mnmajor(u32x4* tile, const T* src, int ld, int c_valid, Perm perm) {
  constexpr int V = Vec<T>::V;
  constexpr int ITEMS = (ROWS / V) * KVN;
  for (int it = threadIdx.x; it < ITEMS; it += NT) {
    const int kv = it % KVN, rb = it / KVN;
    u32x4 in[V], out[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int c = perm(kv, j);
      in[j] = (c < c_valid) ? ld16(src + (size_t)c * ld + rb * V) : u32x4{0, 0, 0, 0};
    }
    transpose_block<T>(in, out);
#pragma unroll
    for (int i = 0; i < V; ++i) tile[lds_slot<ROWS>(kv, rb * V + i)] = out[i];
  }
}

// Contracted-index permutations for stage_mnmajor.
// LinearPerm: vector kv holds indices kv*V .. kv*V + V - 1.
template <int V> struct LinearPerm {
  __device__ __forceinline__ int operator()(int kv, int j) const { return kv * V + j; }
};
// StepPairPerm (bf16 only): the order in which two 16-row accumulator tiles
// (lane group g holds rows 4g..4g+3 of each) become one 32-element MFMA step:
// vector kv = 4s + g holds indices 32s + 4g + {0,1,2,3} and 32s + 16 + 4g + {0,1,2,3}.
struct StepPairPerm {
  __device__ __forceinline__ int operator()(int kv, int j) const {
    const int g = kv & 3;
    return 32 * (kv >> 2) + ((j < 4) ? (4 * g + j) : (16 + 4 * g + j - 4));
  }
};

// The operand vector of MFMA step s built from fp32 accumulator tiles whose
// lane layout is D[4 * (l / 16) + r][l % 16]: bf16 packs tiles 2s and 2s + 1
// (StepPairPerm order); fp32 reuses tile s as is (LinearPerm order).
template <typename T> __device__ __forceinline__ u32x4 acc_to_frag(const floatx4* tiles, int s);
template <> __device__ __forceinline__ u32x4 acc_to_frag<float>(const floatx4* tiles, int s) {
  return __builtin_bit_cast(u32x4, tiles[s]);
}
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// Two floats to bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
// 2^x by the hardware instruction alone: results below 2^-126 flush to zero
// (exp2f adds a rescaling sequence around it to return denormals).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Sum over the 16 lanes of a DPP row (lanes 16k .. 16k + 15), returned to every
// lane of the row: data-parallel moves within the row (swap neighbours, swap
// pairs, reverse each half row, reverse the row) with no LDS traffic.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row_sum16(float v) {
  v += dpp_f<0xB1>(v);    // quad_perm [1, 0, 3, 2]
  v += dpp_f<0x4E>(v);    // quad_perm [2, 3, 0, 1]
  v += dpp_f<0x141>(v);   // row_half_mirror
  v += dpp_f<0x140>(v);   // row_mirror
  return v;
}
template <> __device__ __forceinline__ u32x4 acc_to_frag<bf16>(const floatx4* tiles, int s) {
  const floatx4 a = tiles[2 * s], b = tiles[2 * s + 1];
  return u32x4{pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]), pack_bf16x2(b[0], b[1]), pack_bf16x2(b[2], b[3])};
}
template <typename T> struct AccPerm;
template <> struct AccPerm<float> { typedef LinearPerm<4> type; };
template <> struct AccPerm<bf16> { typedef StepPairPerm type; };

// ---- asynchronous copies to LDS and the waits that order them ---------------------------
// One direct-to-LDS load: each lane's 16 bytes at g land at LDS byte address
// lds + 16 * lane (the LDS address is wave-uniform, taken from M0). Issued as
// inline asm so that the compiler does not track it: its wait insertion would
// otherwise treat every later transpose read of LDS as a possible alias of the
// transfer and wait for all loads in flight. The ring orders these transfers
// explicitly (wait_loads, then a barrier, before a stage is read). M0 is set
// inside the asm; the kernels that use it (GEMM, attention) have no compiler-
// generated M0 use for the asm to disturb.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}

template <int N> __device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Wait until at most `newer` tiles of L loads each (issued after the awaited
// one) are outstanding; the count must be an immediate, so the cases up to
// MAXN are unrolled.
template <int L, int MAXN> __device__ __forceinline__ void wait_loads(int newer) {
  if constexpr (MAXN > 0) {
    if (newer >= MAXN) {
      wait_vmcnt<L * MAXN>();
      return;
    }
    wait_loads<L, MAXN - 1>(newer);
  } else {
    (void)newer;
    wait_vmcnt<0>();
  }
}
// vmcnt(0), other counters left alone, through the builtin: the compiler counts
// it, so register loads issued before it are known complete afterwards.
__device__ __forceinline__ void wait_vmcnt_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// lgkmcnt(0), other counters left alone. Issued through the builtin, not inline
// asm, so that the compiler's own wait insertion knows the reads are complete:
// it then never has to cover the 16 LDS reads of two MFMA steps at once, which
// the 4-bit LGKM counter cannot track, and which makes it wait for all of them.
__device__ __forceinline__ void wait_lds_reads() {
  __builtin_amdgcn_sched_barrier(0);   // keep MFMAs from being scheduled across the wait
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_sched_barrier(0);
}
// Workgroup barrier without the memory fence __syncthreads() implies: the
// fence would wait for every outstanding global load, including the tiles
// prefetched for later iterations. Each wave has already waited for its own
// loads of the tile about to be read (wait_loads) and for its LDS reads of the
// stage about to be refilled (wait_lds_reads).
__device__ __forceinline__ void barrier_no_fence() { asm volatile("s_barrier" ::: "memory"); }

// ---- dropout masks ---------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy
// as 1, 2, 3", SC 2011): ten rounds of two 32 x 32 -> 64-bit products on a
// 4-word counter, the 2-word key bumped by the Weyl constants between rounds.
__device__ __forceinline__ u32x4 philox10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                          uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t hi0 = __umulhi(0xD2511F53u, c0), lo0 = 0xD2511F53u * c0;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c2), lo1 = 0xCD9E8D57u * c2;
    c0 = hi1 ^ c1 ^ k0;
    c2 = hi0 ^ c3 ^ k1;
    c1 = lo1;
    c3 = lo0;
  }
  return u32x4{c0, c1, c2, c3};
}

// Keep bits of a dropout site. Key (seed, micro-batch); `word` = (block << 2) |
// site; a 16-bit value v keeps its element when v >= thr.
//   attention probability (bh, q, k): counter (k >> 2, q >> 1, bh, word), value
//     (k & 1) of output word 2 (q & 1) + ((k >> 1) & 1);
//   element e of an element-wise site: counter (e >> 3, e >> 35, 0, word), value
//     (e & 1) of output word (e >> 1) & 3.
__device__ __forceinline__ uint32_t keep16(uint32_t w, int half, uint32_t thr) {
  return ((half ? (w >> 16) : (w & 0xffffu)) >= thr) ? 1u : 0u;
}
// bit i: probability (q, k4 + i), i < 4, k4 % 4 == 0 (one draw)
__device__ __forceinline__ uint32_t drop_row4(const DropArgs& a, uint32_t bh, int q, int k4) {
  const u32x4 w = philox10((uint32_t)k4 >> 2, (uint32_t)q >> 1, bh, a.word, a.seed, a.mb);
  const uint32_t x = (q & 1) ? w[2] : w[0], y = (q & 1) ? w[3] : w[1];
  return keep16(x, 0, a.thr) | (keep16(x, 1, a.thr) << 1) | (keep16(y, 0, a.thr) << 2) | (keep16(y, 1, a.thr) << 3);
}
// bit i: probability (q4 + i, k), i < 4, q4 % 4 == 0 (two draws)
__device__ __forceinline__ uint32_t drop_col4(const DropArgs& a, uint32_t bh, int q4, int k) {
  const int kb = (k >> 1) & 1, half = k & 1;
  uint32_t bits = 0;
#pragma unroll
  for (int j = 0; j < 2; ++j) {   // queries q4 + 2j + e share the counter of (q4 >> 1) + j
    const u32x4 w = philox10((uint32_t)k >> 2, ((uint32_t)q4 >> 1) + j, bh, a.word, a.seed, a.mb);
    bits |= keep16(kb ? w[1] : w[0], half, a.thr) << (2 * j);
    bits |= keep16(kb ? w[3] : w[2], half, a.thr) << (2 * j + 1);
  }
  return bits;
}
// bit i: element e8 + i, i < 8, e8 % 8 == 0 (one draw)
__device__ __forceinline__ uint32_t drop_elem8(const DropArgs& a, uint64_t e8) {
  const u32x4 w = philox10((uint32_t)(e8 >> 3), (uint32_t)(e8 >> 35), 0u, a.word, a.seed, a.mb);
  uint32_t bits = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) bits |= keep16(w[i >> 1], i & 1, a.thr) << i;
  return bits;
}

}  // namespace paci
