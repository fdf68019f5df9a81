// The PACI stage runtime behind include/paci_stage.h.
//
// One stage of the asynchronous 1F1B pipeline (Alg. 1): a protocol object
// holding the counters (version t, window count c, unresolved forwards q),
// a single fp32 parameter copy, the fp32 gradient accumulator G, the AdamW
// moments, and an activation store of micro-batch slots. All of it is
// sub-allocated from one caller-owned device arena. Forward, backward and
// step enqueue the hand-written kernels on one in-order HIP stream. Stream
// order alone guards the buffers. The update runs after the K-th backward's
// gradient kernels. The next forward reads the refreshed bf16 weights after
// the update.
//
// Weight gradients follow Alg. 1's accumulate step by default: every backward
// adds its G_W += dY^T X products into the fp32 accumulator right away, so the
// store keeps delay + 1 activation slots, the in-flight count of the paper's
// memory model (appendix "Memory and synchronization properties"). The slot of
// mb is reused by F(mb + delay + 1), which the admission rule lets run only
// after B(mb).
//
// Optional windowed weight gradients (paci_shapes.window = 1; bf16 stages whose
// micro-batch token count is a multiple of 64): each backward keeps its output
// gradients (dqkv, dx1, du, dy of every block) in a per-window buffer, and the K
// micro-batches' G_W += dY^T X products run as one long contraction per weight
// before the update (or before G is read, loaded or the counters reset). The
// sum is the same; G is read-modified once per window instead of once per
// micro-batch. The saved activations X then have to outlive the window: the
// store keeps K + delay slots; the slot of mb is reused by F(mb + K + delay),
// which the protocol admits only after the update that closes mb's window.
//
// Drift semantics (Eq. 1): a backward differentiates the activations saved by
// its forward but reads the current parameters. dgrad uses the current bf16
// weights and LayerNorm backward the current fp32 gammas. Every activation
// that depends on parameters (LN outputs, qkv, attention output, x1, u, a) is
// saved at forward time, never recomputed.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "paci_stage.h"

// ============================================================================================
// Protocol (Alg. 1)
// ============================================================================================
struct paci_fsm {
  int K, delay, t, c, q, next_f, next_b;
};

// HIP status of the last failed call that had no handle to record it in (init).
static int g_init_hip_error = 0;

// ---- static scratch of the allocation-free backward ----------------------------------------
// paci_stage_backward_static takes the attention backward's per-query (lse2, D)
// pairs from this array instead of the stage arena. Each GPU the library runs
// on holds its own copy until the process ends. In host code the name is only a
// stand-in: kernels get the device address that hipGetSymbolAddress returns for
// the current device, looked up once per device by static_scratch().
constexpr size_t kStaticScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device.
hipError_t static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}
}  // namespace

static int fsm_check_forward(const paci_fsm& f, int mb) {
  if (f.c == f.K) return PACI_E_STEP_PENDING;
  if (mb != f.next_f) return PACI_E_ORDER;
  if (!(f.q <= f.delay)) return PACI_E_BACKPRESSURE;  // admission: q_i <= N - i
  return PACI_OK;
}
static int fsm_check_backward(const paci_fsm& f, int mb) {
  if (f.c == f.K) return PACI_E_STEP_PENDING;
  if (mb != f.next_b || f.next_b >= f.next_f) return PACI_E_ORDER;
  return PACI_OK;
}
static int fsm_commit_forward(paci_fsm& f) {
  f.next_f++;
  f.q++;
  return f.t;
}
static int fsm_commit_backward(paci_fsm& f) {
  f.next_b++;
  f.c++;
  f.q--;
  return f.t;
}
static void fsm_commit_step(paci_fsm& f) {
  f.c = 0;
  f.t++;
}
static void fsm_counters(const paci_fsm& f, paci_counters* o) {
  o->version = f.t;
  o->c = f.c;
  o->q = f.q;
  o->next_f = f.next_f;
  o->next_b = f.next_b;
  o->K = f.K;
  o->delay = f.delay;
}

extern "C" int paci_fsm_create(int K, int delay, paci_fsm** out) {
  if (!out || K < 1 || delay < 0) return PACI_E_INVAL;
  paci_fsm* f = new (std::nothrow) paci_fsm{K, delay, 0, 0, 0, 0, 0};
  if (!f) return PACI_E_NOMEM;
  *out = f;
  return PACI_OK;
}
extern "C" int paci_fsm_forward(paci_fsm* f, int mb, int* version) {
  if (!f) return PACI_E_INVAL;
  const int e = fsm_check_forward(*f, mb);
  if (e) return e;
  const int t = fsm_commit_forward(*f);
  if (version) *version = t;
  return PACI_OK;
}
extern "C" int paci_fsm_backward(paci_fsm* f, int mb, int* version) {
  if (!f) return PACI_E_INVAL;
  const int e = fsm_check_backward(*f, mb);
  if (e) return e;
  const int t = fsm_commit_backward(*f);
  if (version) *version = t;
  return f->c == f->K ? PACI_STEP_DUE : PACI_OK;
}
extern "C" int paci_fsm_step(paci_fsm* f, int* new_version) {
  if (!f) return PACI_E_INVAL;
  if (f->c != f->K) return PACI_E_NOT_DUE;
  fsm_commit_step(*f);
  if (new_version) *new_version = f->t;
  return PACI_OK;
}
extern "C" int paci_fsm_counters(const paci_fsm* f, paci_counters* out) {
  if (!f || !out) return PACI_E_INVAL;
  fsm_counters(*f, out);
  return PACI_OK;
}
extern "C" int paci_fsm_destroy(paci_fsm* f) {
  delete f;
  return PACI_OK;
}

extern "C" int paci_schedule(int M, int K, int delay, int32_t* kinds, int32_t* idx, int cap, int* n) {
  if (M < 0 || K < 1 || delay < 0 || !n) return PACI_E_INVAL;
  const int total = 2 * M + M / K;
  *n = total;
  if (cap < total || (total > 0 && (!kinds || !idx))) return PACI_E_INVAL;
  int e = 0;
  auto emit = [&](int k, int i) { kinds[e] = k; idx[e] = i; ++e; };
  for (int i = 0; i < std::min(delay + 1, M); ++i) emit(0, i);
  for (int j = 0; j < M; ++j) {
    emit(1, j);
    if ((j + 1) % K == 0) emit(2, -1);
    if (j + delay + 1 < M) emit(0, j + delay + 1);
  }
  return PACI_OK;
}

extern "C" int paci_schedule_flush(int M, int K, int delay, int32_t* kinds, int32_t* idx, int cap, int* n) {
  if (M < 0 || K < 1 || delay < 0 || !n) return PACI_E_INVAL;
  const int total = 2 * M + M / K;
  *n = total;
  if (cap < total || (total > 0 && (!kinds || !idx))) return PACI_E_INVAL;
  int e = 0;
  auto emit = [&](int k, int i) { kinds[e] = k; idx[e] = i; ++e; };
  // window by window; a window's forwards wait for the previous window's update
  for (int a = 0; a < M; a += K) {
    const int b = std::min(M, a + K);
    for (int i = a; i < std::min(a + delay + 1, b); ++i) emit(0, i);
    for (int j = a; j < b; ++j) {
      emit(1, j);
      if (j + delay + 1 < b) emit(0, j + delay + 1);
    }
    if (b - a == K) emit(2, -1);
  }
  return PACI_OK;
}

// ============================================================================================
// Parameter layout
// ============================================================================================
namespace {

struct TensorRef {
  char name[32];
  int rows, cols;
  int64_t off, numel;
  bool decay;
};

struct BlockRefs {
  int64_t ln1_g, ln1_b, w_qkv, b_qkv, w_o, b_o, ln2_g, ln2_b, w_1, b_1, w_2, b_2;
};

struct ParamTable {
  std::vector<TensorRef> t;
  std::vector<BlockRefs> blocks;
  int64_t wte = -1, wpe = -1, lnf_g = -1, lnf_b = -1, w_lm = -1;
  int64_t total = 0;

  int64_t add(const std::string& name, int rows, int cols, bool decay) {
    TensorRef r;
    memset(r.name, 0, sizeof(r.name));
    strncpy(r.name, name.c_str(), sizeof(r.name) - 1);
    r.rows = rows;
    r.cols = cols;
    r.off = total;
    r.numel = (int64_t)rows * cols;
    r.decay = decay;
    t.push_back(r);
    total += r.numel;
    return r.off;
  }
};

int validate_shapes(const paci_shapes* s, int K, int delay) {
  if (!s) return PACI_E_INVAL;
  if (K < 1 || delay < 0) return PACI_E_INVAL;
  if (s->n_layers < 1 || s->n_heads < 1 || s->head_dim < 1 || s->seq < 1 || s->micro_batch < 1 || s->d_ff < 1)
    return PACI_E_INVAL;
  if (s->d_model != s->n_heads * s->head_dim) return PACI_E_INVAL;
  if (s->kind != PACI_MIDDLE && s->kind != PACI_FIRST && s->kind != PACI_LAST) return PACI_E_UNSUPPORTED;
  if (s->dtype != PACI_FP32 && s->dtype != PACI_BF16) return PACI_E_UNSUPPORTED;
  if (s->recompute != 0 && s->recompute != 1) return PACI_E_INVAL;
  if (s->fused_head != 0 && s->fused_head != 1) return PACI_E_INVAL;
  if (s->window != 0 && s->window != 1) return PACI_E_INVAL;
  if (!(s->dropout >= 0.f && s->dropout < 1.f)) return PACI_E_INVAL;
  if (s->fused_head) {
    if (s->kind != PACI_LAST || s->dtype != PACI_BF16 || s->d_model % 8) return PACI_E_UNSUPPORTED;
    if (delay != 0) return PACI_E_INVAL;   // the recomputed logits must see the forward's parameters
  }
  if (s->lr_warmup < 0 || s->lr_total < 0 || (s->lr_total > 0 && s->lr_warmup > s->lr_total) ||
      !(s->lr_min_ratio >= 0.f && s->lr_min_ratio <= 1.f))
    return PACI_E_INVAL;
  if (s->kind != PACI_MIDDLE && s->vocab < 1) return PACI_E_INVAL;
  if (s->kind == PACI_FIRST && (s->max_pos < 1 || s->seq > s->max_pos)) return PACI_E_INVAL;
  const int dh = s->head_dim;
  if (dh != 32 && dh != 64 && dh != 128) return PACI_E_UNSUPPORTED;
  if (s->dtype == PACI_FP32 && dh == 128) return PACI_E_UNSUPPORTED;
  if (s->d_model % 32 || s->d_ff % 32) return PACI_E_UNSUPPORTED;
  if (s->d_model > 4096 || (s->dtype == PACI_FP32 && s->d_model > 2048)) return PACI_E_UNSUPPORTED;
  const int64_t T = (int64_t)s->micro_batch * s->seq;
  if (T > (1LL << 30)) return PACI_E_UNSUPPORTED;
  if (s->window && (s->recompute || s->dtype != PACI_BF16 || T % 64 || s->d_model % 8 || s->d_ff % 8))
    return PACI_E_UNSUPPORTED;   // the windowed contraction: stored bf16 activations in 64-row segments
  return PACI_OK;
}

ParamTable build_params(const paci_shapes& s) {
  ParamTable p;
  const int d = s.d_model, f = s.d_ff;
  if (s.kind == PACI_FIRST) {
    p.wte = p.add("wte", s.vocab, d, false);
    p.wpe = p.add("wpe", s.max_pos, d, false);
  }
  for (int l = 0; l < s.n_layers; ++l) {
    const std::string h = "h" + std::to_string(l) + ".";
    BlockRefs b;
    b.ln1_g = p.add(h + "ln1_g", d, 1, false);
    b.ln1_b = p.add(h + "ln1_b", d, 1, false);
    b.w_qkv = p.add(h + "w_qkv", 3 * d, d, true);
    b.b_qkv = p.add(h + "b_qkv", 3 * d, 1, false);
    b.w_o = p.add(h + "w_o", d, d, true);
    b.b_o = p.add(h + "b_o", d, 1, false);
    b.ln2_g = p.add(h + "ln2_g", d, 1, false);
    b.ln2_b = p.add(h + "ln2_b", d, 1, false);
    b.w_1 = p.add(h + "w_1", f, d, true);
    b.b_1 = p.add(h + "b_1", f, 1, false);
    b.w_2 = p.add(h + "w_2", d, f, true);
    b.b_2 = p.add(h + "b_2", d, 1, false);
    p.blocks.push_back(b);
  }
  if (s.kind == PACI_LAST) {
    p.lnf_g = p.add("lnf_g", d, 1, false);
    p.lnf_b = p.add("lnf_b", d, 1, false);
    p.w_lm = p.add("w_lm", s.vocab, d, true);
  }
  return p;
}

// ---- arena layout ----------------------------------------------------------------------------
struct Bump {
  size_t off = 0;
  size_t take(size_t bytes) {
    off = (off + 255) & ~(size_t)255;
    const size_t r = off;
    off += bytes;
    return r;
  }
};

struct BlockSlot {  // byte offsets inside one activation slot
  size_t x, n1, qkv, o, x1, n2, gu, a, mean1, rstd1, mean2, rstd2, lse2;   // gu = gelu'(u), a = gelu(u)
};

struct Layout {
  int64_t P = 0;          // parameters
  int64_t T = 0;          // tokens per micro-batch
  int64_t ldz = 0;        // logits row stride (last stage)
  size_t theta, G, m, v, theta16, theta16T = 0, chunks, zeros, ctl = 0, guard = 0;
  bool wT = false;             // transposed bf16 block weights kept (theta16T)
  int nchunks = 0, nguard = 0;
  size_t stash, slot_bytes;
  int n_slots = 1;             // activation slots: delay + 1, or K + delay with windowed weight gradients
  bool window = false;         // weight gradients windowed over the K micro-batches of a window
  // bf16 stages without the window: each backward keeps its blocks' output
  // gradients (a window of one micro-batch) and adds all their weight
  // gradients to G in one grouped launch at its end
  bool wdefer = false;
  size_t wgroup = 0;           // problem tables of that launch, one per activation slot (or work slot)
  int wgroup_n = 0, wgroup_tiles = 0;   // problems per table; workgroups of the 256 x 128 launch
  int wgroup_n1 = 0, wgroup_tiles1 = 0; // leading problems on 256 x 256 tiles (their own launch); its workgroups
  // checkpointed stages: each slot holds the stage input only (c_* offsets,
  // c_bytes per slot); one work slot of the full layout takes the activations
  bool recompute = false;
  size_t c_x = 0, c_ids = 0, c_tgt = 0, c_bytes = 0, work = 0;
  std::vector<BlockSlot> blk;  // per block, inside a slot
  struct WinBlock { size_t dqkv, dx1, du, dy; };   // per block: [K * T, width] each
  std::vector<WinBlock> win;
  size_t s_ids = 0, s_tgt = 0, s_y = 0, s_meanf = 0, s_rstdf = 0, s_nf = 0, s_z = 0, s_lse_ce = 0;
  // dropout: the unmasked output gradient of a block (windowed stages), the
  // unmasked x1 gradient, the masked FFN-branch gradient (stages without the
  // window), and the pre-dropout branch output in the forward
  bool dropout = false;
  size_t w_dyu = 0, w_dx1u = 0, w_g2 = 0, w_zdrop = 0;
  // fused LM head: no logits per slot; (max, sum) per row and 64 columns, target logits
  bool fused_head = false;
  int ngroups = 0;
  size_t w_cepart = 0, w_zt = 0;
  // workspace
  size_t w_dyA, w_dyB, w_du, w_dn, w_dx1, w_do, w_dqkv, w_D, w_part, w_dz = 0, w_dnf = 0, w_loss = 0;
  size_t total;
};

constexpr int64_t CHUNK = 4096;   // AdamW elements per workgroup (many small workgroups: a short last round)

// Dropout: a 16-bit Philox value v keeps its element when v >= thr (0: off)
uint32_t drop_threshold(const paci_shapes& s) { return (uint32_t)std::floor((double)s.dropout * 65536.0 + 0.5); }
enum DropSite { SITE_EMBED = 0, SITE_ATTN = 1, SITE_PROJ = 2, SITE_FFN = 3 };

// The AdamW table (paci::adamw): a range entry per CHUNK elements of a tensor, or,
// for the block weight matrices of a stage that keeps them transposed (wT), one
// 64 x 64 tile entry each, which also writes the tile's transposed bf16 values.
// keep_g: the block matrices' G is not cleared by the update (the next window's
// first backward overwrites it).
bool is_block_matrix(const ParamTable& p, int64_t off) {
  for (const BlockRefs& b : p.blocks)
    if (off == b.w_qkv || off == b.w_o || off == b.w_1 || off == b.w_2) return true;
  return false;
}
std::vector<int4> adamw_table(const ParamTable& p, bool wT, bool keep_g) {
  std::vector<int4> v;
  for (const auto& t : p.t) {
    const bool bm = is_block_matrix(p, t.off);
    const int flags = (t.decay ? paci::ADAMW_DECAY : 0) | ((keep_g && bm) ? 0 : paci::ADAMW_CLEAR_G);
    if (wT && bm) {
      for (int r0 = 0; r0 < t.rows; r0 += 64)
        for (int c0 = 0; c0 < t.cols; c0 += 64)
          v.push_back(int4{(int)t.off, (r0 << 16) | c0, flags | paci::ADAMW_TILE, (t.rows << 16) | t.cols});
    } else {
      for (int64_t b = 0; b < t.numel; b += CHUNK)
        v.push_back(int4{(int)(t.off + b), (int)(t.off + std::min(t.numel, b + CHUNK)), flags, 0});
    }
  }
  return v;
}
// Ranges the step's non-finite guard reads when the block matrices' G was
// checked by the last backward of the window: every other tensor, in CHUNK pieces.
std::vector<int2> guard_table(const ParamTable& p) {
  std::vector<int2> v;
  for (const auto& t : p.t)
    if (!is_block_matrix(p, t.off))
      for (int64_t b = 0; b < t.numel; b += CHUNK) v.push_back(int2{(int)(t.off + b), (int)(t.off + std::min(t.numel, b + CHUNK))});
  return v;
}

Layout make_layout(const paci_shapes& s, int K, int delay, const ParamTable& p) {
  Layout L;
  const int64_t esz = s.dtype == PACI_BF16 ? 2 : 4;
  const int64_t d = s.d_model, f = s.d_ff, T = (int64_t)s.micro_batch * s.seq;
  const int64_t heads_rows = (int64_t)s.micro_batch * s.n_heads * s.seq;
  L.P = p.total;
  L.T = T;
  L.ldz = ((int64_t)s.vocab + 63) / 64 * 64;
  Bump a;
  L.theta = a.take(4 * L.P);
  L.G = a.take(4 * L.P);
  L.m = a.take(4 * L.P);
  L.v = a.take(4 * L.P);
  L.theta16 = s.dtype == PACI_BF16 ? a.take(2 * L.P) : 0;
  // bf16 stages: the block weight matrices also transposed ([in, out]), at the
  // same offsets, for the input-gradient GEMMs
  // (tile entries of the AdamW table pack rows and columns in 16 bits each)
  L.wT = s.dtype == PACI_BF16 && d % 8 == 0 && f % 8 == 0 && 3 * d < 32768 && f < 32768;
  L.theta16T = L.wT ? a.take(2 * L.P) : 0;
  L.nchunks = (int)adamw_table(p, L.wT, false).size();
  L.chunks = a.take(16 * (size_t)L.nchunks);
  L.nguard = (int)guard_table(p).size();
  L.guard = a.take(8 * (size_t)std::max(1, L.nguard));
  L.zeros = a.take(256);  // never written after init: source of out-of-range GEMM tile slots
  L.ctl = a.take(256);    // update control: {G not finite, updates applied, updates skipped, 0}

  // one activation slot
  Bump sl;
  for (int l = 0; l < s.n_layers; ++l) {
    BlockSlot b;
    b.x = sl.take(esz * T * d);
    b.n1 = sl.take(esz * T * d);
    b.qkv = sl.take(esz * T * 3 * d);
    b.o = sl.take(esz * T * d);
    b.x1 = sl.take(esz * T * d);
    b.n2 = sl.take(esz * T * d);
    b.gu = sl.take(esz * T * f);
    b.a = sl.take(esz * T * f);
    b.mean1 = sl.take(4 * T);
    b.rstd1 = sl.take(4 * T);
    b.mean2 = sl.take(4 * T);
    b.rstd2 = sl.take(4 * T);
    b.lse2 = sl.take(4 * heads_rows);
    L.blk.push_back(b);
  }
  if (s.kind == PACI_FIRST) L.s_ids = sl.take(4 * T);
  if (s.kind == PACI_LAST) {
    L.s_tgt = sl.take(4 * T);
    L.s_y = sl.take(esz * T * d);
    L.s_meanf = sl.take(4 * T);
    L.s_rstdf = sl.take(4 * T);
    L.s_nf = sl.take(esz * T * d);
    L.fused_head = s.fused_head != 0;
    if (!L.fused_head) L.s_z = sl.take(4 * T * L.ldz);
    L.s_lse_ce = sl.take(4 * T);
  }
  L.slot_bytes = (sl.off + 255) & ~(size_t)255;
  L.recompute = s.recompute != 0;
  L.window = s.window != 0;   // validate_shapes admits it only where the windowed kernels apply
  L.wdefer = !L.window && s.dtype == PACI_BF16 && T % 8 == 0 && d % 8 == 0 && f % 8 == 0;
  L.n_slots = L.window ? K + delay : delay + 1;
  if (L.recompute) {
    Bump c;
    if (s.kind == PACI_FIRST) L.c_ids = c.take(4 * T);
    else L.c_x = c.take(esz * T * d);
    if (s.kind == PACI_LAST) L.c_tgt = c.take(4 * T);
    L.c_bytes = (c.off + 255) & ~(size_t)255;
    L.stash = a.take(L.c_bytes * (size_t)L.n_slots);
    L.work = a.take(L.slot_bytes);
  } else {
    L.stash = a.take(L.slot_bytes * (size_t)L.n_slots);
  }
  if (L.window || L.wdefer) {
    const size_t wk = L.window ? (size_t)K : 1;   // micro-batches per window buffer
    for (int l = 0; l < s.n_layers; ++l) {
      Layout::WinBlock w;
      w.dqkv = a.take(esz * wk * T * 3 * d);
      w.dx1 = a.take(esz * wk * T * d);
      w.du = a.take(esz * wk * T * f);
      w.dy = a.take(esz * wk * T * d);
      L.win.push_back(w);
    }
  }
  if (L.wdefer) {
    L.wgroup_n = 4 * s.n_layers;
    const int tables = L.recompute ? 1 : L.n_slots;
    L.wgroup = a.take(sizeof(paci::WgradProblem) * (size_t)L.wgroup_n * tables);
    // shapes in table order (wgrad_tables): per block W_2, W_1, W_o, W_qkv
    const int shapes[4][2] = {{(int)d, (int)f}, {(int)f, (int)d}, {(int)d, (int)d}, {3 * (int)d, (int)d}};
    std::vector<int> Ms, Ns;
    for (int l = 0; l < s.n_layers; ++l)
      for (int q = 0; q < 4; ++q) {
        Ms.push_back(shapes[q][0]);
        Ns.push_back(shapes[q][1]);
      }
    L.wgroup_n1 = paci::wgrad_group_wide(Ms.data(), Ns.data(), L.wgroup_n);
    int tiles1 = 0, tiles = 0;
    for (int p = 0; p < L.wgroup_n; ++p) {
      const bool wide = p < L.wgroup_n1;
      (wide ? tiles1 : tiles) += (paci::wgrad_group_tiles(Ms[p], Ns[p], wide) + 7) / 8 * 8;
    }
    L.wgroup_tiles1 = tiles1;
    L.wgroup_tiles = tiles;
  }

  // backward workspace (one micro-batch at a time)
  L.w_dyA = a.take(esz * T * d);
  L.w_dyB = a.take(esz * T * d);
  L.w_du = a.take(esz * T * f);
  L.w_dn = a.take(esz * T * d);
  L.w_dx1 = a.take(esz * T * d);
  L.w_do = a.take(esz * T * d);
  L.w_dqkv = a.take(esz * T * 3 * d);
  L.w_D = a.take(4 * (size_t)paci::attn_bwd_workspace_floats(s.dtype == PACI_BF16 ? paci::DT_BF16 : paci::DT_F32,
                                                              s.micro_batch, s.seq, s.n_heads));
  int64_t part = 64;
  if (s.kind == PACI_LAST) {
    part = std::max(part, paci::ce_part_floats((int)T));
    L.w_dz = a.take(esz * T * L.ldz);
    L.w_dnf = a.take(esz * T * d);
    if (L.fused_head) {
      L.ngroups = (int)(L.ldz / 64);
      L.w_cepart = a.take(8 * T * (int64_t)L.ngroups);
      L.w_zt = a.take(4 * T);
    }
  }
  L.w_part = a.take(4 * part);
  L.w_loss = a.take(256);
  L.dropout = drop_threshold(s) > 0;
  if (L.dropout) {
    L.w_dyu = a.take(esz * T * d);
    L.w_dx1u = a.take(esz * T * d);
    L.w_g2 = a.take(esz * T * d);
    L.w_zdrop = a.take(esz * T * d);
  }
  L.total = (a.off + 255) & ~(size_t)255;
  return L;
}

// ---- kernel timing families -------------------------------------------------------------------
enum Family {
  F_GEMM_FWD = 0, F_GEMM_DGRAD, F_GEMM_WGRAD, F_ATTN_FWD, F_ATTN_BWD, F_LN_FWD, F_LN_BWD, F_BIAS_GRAD, F_ADAMW,
  F_EMBED, F_CE, F_COPY, F_DROPOUT, F_COUNT
};
const char* kFamilyNames[F_COUNT] = {"gemm_fwd", "gemm_dgrad", "gemm_wgrad_acc", "attn_fwd", "attn_bwd",
                                     "layernorm_fwd", "layernorm_bwd", "bias_grad", "adamw", "embedding",
                                     "cross_entropy", "copy", "dropout"};

}  // namespace

// ============================================================================================
// The stage handle
// ============================================================================================
struct paci_stage {
  paci_shapes s;
  paci_fsm fsm;
  hipStream_t st;
  char* arena;
  ParamTable p;
  Layout L;
  paci::DType dt;
  int esz;
  int last_hip = 0;
  bool broken = false;
  int win_done = 0;   // micro-batches of the current window whose weight gradients are in G
  // Grouped weight gradients (L.wdefer): after an update the block matrices' G is
  // logically zero but not cleared; the next backward's products overwrite it.
  bool g_lazy = false;
  // the next step guards all of G (else only the ranges of L.guard: the last
  // backward of the window checked the block matrices' G as it wrote it)
  bool guard_full = true;

  // the attention backward's (lse2, D) pairs: the arena's workspace, or (during
  // paci_stage_backward_static) the static scratch of this device
  float* pairs = nullptr;
  void* static_pairs = nullptr;   // device address of `scratch` on the stage's GPU
  bool no_events = false;         // no timing events (they may allocate) during the static variant

  // timing
  bool timing = false;
  struct Pending { hipEvent_t a, b; int fam; double work; };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> free_ev;
  int64_t launches[F_COUNT] = {};
  double ms[F_COUNT] = {}, work[F_COUNT] = {};

  // dropout at one site of micro-batch mb (thr 0 when the stage has none)
  paci::DropArgs drop(int mb, int block, int site) const {
    paci::DropArgs a;
    if (!L.dropout) return a;
    a.seed = s.dropout_seed;
    a.mb = (uint32_t)mb;
    a.word = ((uint32_t)block << 2) | (uint32_t)site;
    a.thr = drop_threshold(s);
    a.scale = 1.f / (1.f - s.dropout);
    return a;
  }
  float* theta() const { return reinterpret_cast<float*>(arena + L.theta); }
  float* G() const { return reinterpret_cast<float*>(arena + L.G); }
  float* m() const { return reinterpret_cast<float*>(arena + L.m); }
  float* v() const { return reinterpret_cast<float*>(arena + L.v); }
  // weights as consumed by the matrix kernels: the bf16 working copy, or fp32 itself
  const void* W(int64_t off) const {
    return dt == paci::DT_BF16 ? (const void*)(reinterpret_cast<const uint16_t*>(arena + L.theta16) + off)
                               : (const void*)(theta() + off);
  }
  // transposed bf16 copy of a block weight matrix [out, in] -> [in, out]
  const void* WT(int64_t off) const { return reinterpret_cast<const uint16_t*>(arena + L.theta16T) + off; }
  const float* th(int64_t off) const { return theta() + off; }
  float* g(int64_t off) const { return G() + off; }
  // the slot of mb: the stage input only on a checkpointed stage, else every activation
  char* slot(int mb) const {
    return arena + L.stash + (size_t)(mb % L.n_slots) * (L.recompute ? L.c_bytes : L.slot_bytes);
  }
  // where a micro-batch's activations are computed: the work slot, or its own slot
  char* acts(int mb) const { return L.recompute ? arena + L.work : slot(mb); }
  // window buffer of block l, tensor at offset off, micro-batch j of the window, width columns
  char* win(size_t off, int j, int width) const { return arena + off + (size_t)j * L.T * width * esz; }
  char* ws(size_t off) const { return arena + off; }
};

namespace {

hipEvent_t take_event(paci_stage* h) {
  if (!h->free_ev.empty()) {
    hipEvent_t e = h->free_ev.back();
    h->free_ev.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void drain_timing(paci_stage* h) {
  for (auto& p : h->pending) {
    float t = 0.f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&t, p.a, p.b) == hipSuccess) {
      h->launches[p.fam]++;
      h->ms[p.fam] += t;
      h->work[p.fam] += p.work;
    }
    h->free_ev.push_back(p.a);
    h->free_ev.push_back(p.b);
  }
  h->pending.clear();
}

// Runs one launch, bracketed by events when timing is on. Returns a PACI status.
template <class F>
int run(paci_stage* h, int fam, double work, F&& launch) {
  hipEvent_t a = nullptr, b = nullptr;
  if (h->timing && !h->no_events) {
    if (h->pending.size() >= 65536) drain_timing(h);  // bounded pool; drains synchronize
    a = take_event(h);
    b = take_event(h);
    if (a && b) (void)hipEventRecord(a, h->st);
  }
  const hipError_t e = launch();
  if (e != hipSuccess) {
    h->last_hip = (int)e;
    h->broken = true;
    return PACI_E_HIP;
  }
  if (h->timing && !h->no_events && a && b) {
    (void)hipEventRecord(b, h->st);
    h->pending.push_back({a, b, fam, work});
  }
  return PACI_OK;
}

#define TRY(x)                 \
  do {                         \
    const int _r = (x);        \
    if (_r != PACI_OK) return _r; \
  } while (0)

// ---- linear-layer helpers -------------------------------------------------------------------
int linear_fwd(paci_stage* h, const void* X, int64_t w_off, int64_t b_off, int M, int N, int K, paci::GemmEpi epi,
               void* C, const void* aux, void* C2) {
  paci::GemmArgs a{X, K, h->W(w_off), K, M, N, K, C, N, b_off >= 0 ? h->th(b_off) : nullptr, aux, N, C2,
                   h->arena + h->L.zeros};
  return run(h, F_GEMM_FWD, 2.0 * M * N * K,
             [&] { return paci::gemm(h->dt, false, paci::GEMM_NT, epi, a, 1, h->st); });
}

// dX [M, N] = dY [M, K] . W [K, N]   (W = nn.Linear weight [out = K, in = N])
// colsum_off >= 0: also accumulate the column sums of dX into that gradient.
// block: W is a block weight, so with transposed copies kept the product reads
// W^T [N, K] and both operands are contiguous along K.
int linear_dgrad(paci_stage* h, const void* dY, int64_t ldy, int64_t w_off, int M, int N, int K, paci::GemmEpi epi,
                 void* C, const void* aux, int64_t colsum_off = -1, bool block = true) {
  const bool tr = block && h->L.wT;
  paci::GemmArgs a{dY, ldy, tr ? h->WT(w_off) : h->W(w_off), tr ? K : N, M, N, K, C, N, nullptr, aux, N, nullptr,
                   h->arena + h->L.zeros};
  if (colsum_off >= 0) a.colsum = h->g(colsum_off);
  return run(h, F_GEMM_DGRAD, 2.0 * M * N * K,
             [&] { return paci::gemm(h->dt, false, tr ? paci::GEMM_NT : paci::GEMM_NN, epi, a, 1, h->st); });
}

// Rewrites the transposed bf16 block weights from the bf16 working copy.
int refresh_wT(paci_stage* h) {
  if (!h->L.wT) return PACI_OK;
  const int d = h->s.d_model, f = h->s.d_ff;
  const uint16_t* w16 = reinterpret_cast<const uint16_t*>(h->arena + h->L.theta16);
  uint16_t* wt = reinterpret_cast<uint16_t*>(h->arena + h->L.theta16T);
  for (const BlockRefs& b : h->p.blocks) {
    const int64_t offs[4] = {b.w_qkv, b.w_o, b.w_1, b.w_2};
    const int rows[4] = {3 * d, d, f, d}, cols[4] = {d, d, d, f};
    for (int i = 0; i < 4; ++i)
      TRY(run(h, F_ADAMW, 4.0 * rows[i] * cols[i],
              [&] { return paci::transpose16(w16 + offs[i], wt + offs[i], rows[i], cols[i], h->st); }));
  }
  return PACI_OK;
}

// G[out, in] += dY[T, out]^T X[T, in]
int linear_wgrad(paci_stage* h, const void* dY, int64_t ldy, const void* X, int64_t ldx, int out, int in, int T,
                 int64_t g_off) {
  const int splits = paci::gemm_acc_splits(h->dt, out, in, T);
  paci::GemmArgs a{dY, ldy, X, ldx, out, in, T, h->g(g_off), in, nullptr, nullptr, 0, nullptr, h->arena + h->L.zeros};
  const paci::GemmEpi epi = splits > 1 ? paci::EPI_ATOMIC : paci::EPI_ACC;
  return run(h, F_GEMM_WGRAD, 2.0 * out * in * T,
             [&] { return paci::gemm(h->dt, true, paci::GEMM_TN, epi, a, splits, h->st); });
}

int bias_grad(paci_stage* h, const void* Y, int64_t ld, int rows, int ncols, int64_t g_off) {
  return run(h, F_BIAS_GRAD, (double)rows * ncols * h->esz, [&] {
    return paci::colsum_acc(h->dt, Y, ld, rows, ncols, h->g(g_off), h->st);
  });
}

// out = res + z * keep * scale over [T, d] (res nullable)
int dropout(paci_stage* h, const void* z, const void* res, void* out, const paci::DropArgs& a) {
  const int T = (int)h->L.T, d = h->s.d_model;
  return run(h, F_DROPOUT, (double)T * d * h->esz * (res ? 3 : 2),
             [&] { return paci::dropout_fwd(h->dt, z, res, out, T, d, a, h->st); });
}

int ln_fwd(paci_stage* h, const void* x, void* n, float* mean, float* rstd, int64_t g_off, int64_t b_off,
           void* xcopy) {
  const int T = (int)h->L.T, d = h->s.d_model;
  return run(h, F_LN_FWD, (double)T * d * 2 * h->esz + 8.0 * T, [&] {
    return paci::layernorm_fwd(h->dt, x, n, mean, rstd, h->th(g_off), h->th(b_off), xcopy, T, d, h->s.ln_eps, h->st);
  });
}

// gd_off >= 0: also accumulate sum_rows dx into that gradient (the output-bias
// gradient of the linear layer that produced x, or of the block before)
int ln_bwd(paci_stage* h, const void* dn, const void* x, const float* mean, const float* rstd, int64_t g_off,
           int64_t b_off, const void* res, void* dx, int64_t gd_off = -1) {
  const int T = (int)h->L.T, d = h->s.d_model;
  // dx pass (dn, x, res in, dx out) and column pass (dn, x and, for gd_off, dx again)
  return run(h, F_LN_BWD, (double)T * d * ((res ? 4 : 3) + 2 + (gd_off >= 0 ? 1 : 0)) * h->esz + 8.0 * T, [&] {
    return paci::layernorm_bwd(h->dt, dn, x, mean, rstd, h->th(g_off), res, dx, h->g(g_off), h->g(b_off),
                               gd_off >= 0 ? h->g(gd_off) : nullptr, T, d, h->st);
  });
}

double attn_pairs(const paci_shapes& s) {
  return (double)s.micro_batch * s.n_heads * ((double)s.seq * (s.seq + 1) / 2.0);
}

// ---- forward of the block stack -----------------------------------------------------------------
// in: block-0 input (stage input or embedding output); x0_copy: where to store a
// copy of it (nullptr: `in` stays valid), which block 0's residual then reads.
int blocks_fwd(paci_stage* h, char* sl, const void* in, void* x0_copy, void* out, int mb) {
  const paci_shapes& s = h->s;
  const int T = (int)h->L.T, d = s.d_model, f = s.d_ff;
  for (int l = 0; l < s.n_layers; ++l) {
    const BlockRefs& b = h->p.blocks[l];
    const BlockSlot& o = h->L.blk[l];
    const void* x = (l == 0) ? in : (const void*)(sl + o.x);
    float* mean1 = reinterpret_cast<float*>(sl + o.mean1);
    float* rstd1 = reinterpret_cast<float*>(sl + o.rstd1);
    TRY(ln_fwd(h, x, sl + o.n1, mean1, rstd1, b.ln1_g, b.ln1_b, l == 0 ? x0_copy : nullptr));
    TRY(linear_fwd(h, sl + o.n1, b.w_qkv, b.b_qkv, T, 3 * d, d, paci::EPI_BIAS, sl + o.qkv, nullptr, nullptr));
    TRY(run(h, F_ATTN_FWD, 4.0 * attn_pairs(s) * s.head_dim, [&] {
      return paci::attn_fwd(h->dt, sl + o.qkv, sl + o.o, reinterpret_cast<float*>(sl + o.lse2), s.micro_batch, s.seq,
                            s.n_heads, s.head_dim, h->drop(mb, l, SITE_ATTN), h->st);
    }));
    const void* res = l > 0 ? (const void*)(sl + o.x) : (x0_copy ? (const void*)x0_copy : in);
    char* zd = h->L.dropout ? h->ws(h->L.w_zdrop) : nullptr;   // a branch output before its dropout
    if (zd) {
      TRY(linear_fwd(h, sl + o.o, b.w_o, b.b_o, T, d, d, paci::EPI_BIAS, zd, nullptr, nullptr));
      TRY(dropout(h, zd, res, sl + o.x1, h->drop(mb, l, SITE_PROJ)));
    } else {
      TRY(linear_fwd(h, sl + o.o, b.w_o, b.b_o, T, d, d, paci::EPI_BIAS_RES, sl + o.x1, res, nullptr));
    }
    TRY(ln_fwd(h, sl + o.x1, sl + o.n2, reinterpret_cast<float*>(sl + o.mean2), reinterpret_cast<float*>(sl + o.rstd2),
               b.ln2_g, b.ln2_b, nullptr));
    TRY(linear_fwd(h, sl + o.n2, b.w_1, b.b_1, T, f, d, paci::EPI_BIAS_GELU, sl + o.gu, nullptr, sl + o.a));
    void* y = (l + 1 < s.n_layers) ? (void*)(sl + h->L.blk[l + 1].x) : out;
    if (zd) {
      TRY(linear_fwd(h, sl + o.a, b.w_2, b.b_2, T, d, f, paci::EPI_BIAS, zd, nullptr, nullptr));
      TRY(dropout(h, zd, sl + o.x1, y, h->drop(mb, l, SITE_FFN)));
    } else {
      TRY(linear_fwd(h, sl + o.a, b.w_2, b.b_2, T, d, f, paci::EPI_BIAS_RES, y, sl + o.x1, nullptr));
    }
  }
  return PACI_OK;
}

// ---- backward of one block: dy -> dx ------------------------------------------------------------
// dy_bias_done: G_b2 of this block already holds sum dy (accumulated by the
// LayerNorm backward that produced dy)
// j: the micro-batch's position in its window (windowed weight gradients: the
// block's output gradients go to the window buffer and G_W waits for the flush)
int block_bwd(paci_stage* h, char* sl, int l, const void* dy, void* dx, bool dy_bias_done, int j, int mb) {
  const paci_shapes& s = h->s;
  const int T = (int)h->L.T, d = s.d_model, f = s.d_ff;
  const BlockRefs& b = h->p.blocks[l];
  const BlockSlot& o = h->L.blk[l];
  const Layout& L = h->L;
  const bool win = L.window || L.wdefer, drop = L.dropout;
  char* du = win ? h->win(L.win[l].du, j, f) : h->ws(L.w_du);
  char* dn = h->ws(L.w_dn);
  char* dx1 = win ? h->win(L.win[l].dx1, j, d) : h->ws(L.w_dx1);
  char* dO = h->ws(L.w_do);
  char* dqkv = win ? h->win(L.win[l].dqkv, j, 3 * d) : h->ws(L.w_dqkv);
  // y = x1 + drop(a W2^T + b2): the branch gets g2 = dy * keep * scale (without
  // dropout g2 = dy); the residual path keeps dy. A windowed stage's window
  // slot must end up holding g2 (the flush contracts it), so dy moves aside.
  const void* dyu = dy;
  const void* g2 = dy;
  if (drop) {
    char* g2buf = win ? h->win(L.win[l].dy, j, d) : h->ws(L.w_g2);
    if (win) {
      TRY(run(h, F_COPY, 2.0 * T * d * h->esz, [&] {
        return hipMemcpyAsync(h->ws(L.w_dyu), dy, (size_t)T * d * h->esz, hipMemcpyDeviceToDevice, h->st);
      }));
      dyu = h->ws(L.w_dyu);
    }
    TRY(dropout(h, dyu, nullptr, g2buf, h->drop(mb, l, SITE_FFN)));
    g2 = g2buf;
  }
  if (!win) TRY(linear_wgrad(h, g2, d, sl + o.a, f, d, f, T, b.w_2));
  if (!dy_bias_done || drop) TRY(bias_grad(h, g2, d, T, d, b.b_2));
  // du = (g2 W2) * gelu'(u) (kept by the forward), and G_b1 += sum du in the same epilogue
  TRY(linear_dgrad(h, g2, d, b.w_2, T, f, d, paci::EPI_GELU_GRAD, du, sl + o.gu, b.b_1));
  // u = n2 W1^T + b1
  if (!win) TRY(linear_wgrad(h, du, f, sl + o.n2, d, f, d, T, b.w_1));
  TRY(linear_dgrad(h, du, f, b.w_1, T, d, f, paci::EPI_STORE, dn, nullptr));
  // n2 = LN2(x1); dL/dx1 = dy + LN2 backward (and G_bo += its column sums when
  // there is no dropout: then it is also the projection branch's gradient)
  char* dx1u = drop ? h->ws(L.w_dx1u) : dx1;
  TRY(ln_bwd(h, dn, sl + o.x1, reinterpret_cast<const float*>(sl + o.mean2),
             reinterpret_cast<const float*>(sl + o.rstd2), b.ln2_g, b.ln2_b, dyu, dx1u, drop ? -1 : b.b_o));
  // x1 = x + drop(o Wo^T + bo): the branch gets g1 = dL/dx1 * keep * scale, in dx1
  if (drop) {
    TRY(dropout(h, dx1u, nullptr, dx1, h->drop(mb, l, SITE_PROJ)));
    TRY(bias_grad(h, dx1, d, T, d, b.b_o));
  }
  if (!win) TRY(linear_wgrad(h, dx1, d, sl + o.o, d, d, d, T, b.w_o));
  TRY(linear_dgrad(h, dx1, d, b.w_o, T, d, d, paci::EPI_STORE, dO, nullptr));
  // attention; G_bqkv += sum dqkv in the same kernels
  TRY(run(h, F_ATTN_BWD, 8.0 * attn_pairs(s) * s.head_dim, [&] {
    return paci::attn_bwd(h->dt, sl + o.qkv, sl + o.o, dO, reinterpret_cast<const float*>(sl + o.lse2),
                          h->pairs, dqkv, h->g(b.b_qkv), s.micro_batch, s.seq,
                          s.n_heads, s.head_dim, h->drop(mb, l, SITE_ATTN), h->st);
  }));
  // qkv = n1 Wqkv^T + bqkv
  if (!win) TRY(linear_wgrad(h, dqkv, 3 * d, sl + o.n1, d, 3 * d, d, T, b.w_qkv));
  TRY(linear_dgrad(h, dqkv, 3 * d, b.w_qkv, T, d, 3 * d, paci::EPI_STORE, dn, nullptr));
  // n1 = LN1(x); dx = dL/dx1 + LN1 backward; dx is the output gradient of block
  // l - 1, so (without dropout) G_b2 of that block += sum dx
  TRY(ln_bwd(h, dn, sl + o.x, reinterpret_cast<const float*>(sl + o.mean1),
             reinterpret_cast<const float*>(sl + o.rstd1), b.ln1_g, b.ln1_b, dx1u, dx,
             (l > 0 && !drop) ? h->p.blocks[l - 1].b_2 : -1));
  return PACI_OK;
}

size_t act_bytes(const paci_stage* h) { return (size_t)h->L.T * h->s.d_model * h->esz; }

// G[out, in] += dY^T X over micro-batches j0 .. j0 + n - 1 of the window: dY from the
// window buffer (contiguous), X from the activation slots of those micro-batches
// (first micro-batch mb0), one contracted segment of T rows per slot.
// Split-K count for these long contractions (256 x 128 output tiles, one
// workgroup per CU): about 512 workgroups, two rounds over the CUs, each split
// at least 1024 contracted rows, at most 16 splits (measured on MI355X for
// 64K-row weight gradients at d = 1024: 512 beat 768 and 1024).
int window_splits(int out, int in, int64_t Kt) {
  const int64_t tiles = (int64_t)((out + 255) / 256) * ((in + 127) / 128);
  const int by_rows = (int)std::min<int64_t>(16, Kt / 1024);
  return std::max(1, std::min(by_rows, (int)std::lround(512.0 / (double)tiles)));
}

int window_wgrad(paci_stage* h, size_t dy_off, size_t x_off, int out, int in, int j0, int n, int mb0,
                 int64_t g_off) {
  const Layout& L = h->L;
  const int64_t Kt = (int64_t)n * L.T;
  const int splits = window_splits(out, in, Kt);
  paci::GemmArgs a{h->win(dy_off, j0, out), out, h->arena + L.stash + x_off, in, out, in, (int)Kt, h->g(g_off), in,
                   nullptr, nullptr, 0, nullptr, h->arena + L.zeros};
  a.seg_rows = L.T;
  a.seg_stride = (int64_t)(L.slot_bytes / (size_t)h->esz);
  a.seg_first = mb0 % L.n_slots;
  a.seg_count = L.n_slots;
  const paci::GemmEpi epi = splits > 1 ? paci::EPI_ATOMIC : paci::EPI_ACC;
  return run(h, F_GEMM_WGRAD, 2.0 * out * in * (double)Kt,
             [&] { return paci::gemm(h->dt, true, paci::GEMM_TN, epi, a, splits, h->st); });
}

// Adds the weight gradients of the window's micro-batches not yet in G (Alg. 1
// accumulates them per backward; the sum is the same).
int flush_window(paci_stage* h) {
  const Layout& L = h->L;
  if (!L.window) return PACI_OK;
  const int c = h->fsm.c, j0 = h->win_done;
  if (c <= j0) return PACI_OK;
  const int n = c - j0, mb0 = h->fsm.next_b - c + j0;
  const int d = h->s.d_model, f = h->s.d_ff;
  for (int l = 0; l < h->s.n_layers; ++l) {
    const BlockRefs& b = h->p.blocks[l];
    const BlockSlot& o = L.blk[l];
    const Layout::WinBlock& w = L.win[l];
    TRY(window_wgrad(h, w.dy, o.a, d, f, j0, n, mb0, b.w_2));
    TRY(window_wgrad(h, w.du, o.n2, f, d, j0, n, mb0, b.w_1));
    TRY(window_wgrad(h, w.dx1, o.o, d, d, j0, n, mb0, b.w_o));
    TRY(window_wgrad(h, w.dqkv, o.n1, 3 * d, d, j0, n, mb0, b.w_qkv));
  }
  h->win_done = c;
  return PACI_OK;
}

// The weight gradients of every block of one backward, from the output
// gradients it left in the window buffers and the activations of its slot
// (table t), in one grouped launch: G_W += dY^T X for the four weights of each
// block (Alg. 1's accumulate step for this backward).
// overwrite: the block matrices' G is logically zero (after an update), so the
// products are stored instead of added; flag: the window's last backward sets
// the non-finite flag of the update control words if any sum it writes is not finite.
int wgrad_grouped(paci_stage* h, int t, bool overwrite, int* flag) {
  const Layout& L = h->L;
  const double T = (double)L.T, d = h->s.d_model, f = h->s.d_ff;
  const double work = 2.0 * T * h->s.n_layers * (d * f + f * d + d * d + 3 * d * d);
  const auto* tab = reinterpret_cast<const paci::WgradProblem*>(h->arena + L.wgroup) + (size_t)t * L.wgroup_n;
  const int n1 = L.wgroup_n1;
  return run(h, F_GEMM_WGRAD, work, [&] {
    // the leading problems on 256 x 256 tiles, the rest on 256 x 128 (each launch
    // fills whole rounds of the CUs where the shapes allow)
    hipError_t e = hipSuccess;
    if (n1 > 0)
      e = paci::gemm_wgrad_grouped(tab, n1, L.wgroup_tiles1, (int)L.T, h->arena + L.zeros, overwrite, true, flag,
                                   h->st);
    if (e == hipSuccess && n1 < L.wgroup_n)
      e = paci::gemm_wgrad_grouped(tab + n1, L.wgroup_n - n1, L.wgroup_tiles, (int)L.T, h->arena + L.zeros,
                                   overwrite, false, flag, h->st);
    return e;
  });
}

// Makes a logically zero G of the block matrices zero in memory (before G is read).
int materialize_g(paci_stage* h) {
  if (!h->g_lazy) return PACI_OK;
  for (const auto& t : h->p.t)
    if (is_block_matrix(h->p, t.off))
      TRY(run(h, F_COPY, 4.0 * (double)t.numel, [&] { return paci::fill_f32(h->g(t.off), t.numel, 0.f, h->st); }));
  h->g_lazy = false;
  return PACI_OK;
}

// Problem tables of the grouped launch, one per activation area a backward can read.
std::vector<paci::WgradProblem> wgrad_tables(const paci_stage* h) {
  const Layout& L = h->L;
  const int d = h->s.d_model, f = h->s.d_ff;
  const int tables = L.recompute ? 1 : L.n_slots;
  std::vector<paci::WgradProblem> v;
  for (int t = 0; t < tables; ++t) {
    const char* A = L.recompute ? h->arena + L.work : h->arena + L.stash + (size_t)t * L.slot_bytes;
    int tile0 = 0, p = 0;   // tile0 restarts at the first problem of the 256 x 128 launch
    for (int l = h->s.n_layers - 1; l >= 0; --l) {   // the order the backward produced them
      const BlockRefs& b = h->p.blocks[l];
      const BlockSlot& o = L.blk[l];
      const Layout::WinBlock& w = L.win[l];
      const struct { size_t dy, x; int M, N; int64_t g; } q[4] = {
          {w.dy, o.a, d, f, b.w_2}, {w.du, o.n2, f, d, b.w_1}, {w.dx1, o.o, d, d, b.w_o}, {w.dqkv, o.n1, 3 * d, d, b.w_qkv}};
      for (const auto& e : q) {
        const bool wide = p < L.wgroup_n1;
        if (p++ == L.wgroup_n1) tile0 = 0;
        paci::WgradProblem pr;
        pr.A = h->arena + e.dy;
        pr.B = A + e.x;
        pr.C = h->G() + e.g;
        pr.M = e.M;
        pr.N = e.N;
        pr.tile0 = tile0;
        pr.xcd_m = paci::wgrad_group_xcd_m(e.M, e.N, (int)L.T, wide);
        v.push_back(pr);
        tile0 += (paci::wgrad_group_tiles(e.M, e.N, wide) + 7) / 8 * 8;
      }
    }
  }
  return v;
}

// The stage forward of one micro-batch into the activation area A (its slot, or
// the work slot of a checkpointed stage). in: the stage input (middle, last);
// x0_copy: where block 0 keeps it; ids / tgt: the micro-batch's token ids (first
// stage) and targets (last stage) as stored; out: the stage output (last stage:
// the loss).
int stage_forward_into(paci_stage* h, char* A, const void* in, void* x0_copy, const int32_t* ids,
                       const int32_t* tgt, void* out, int mb) {
  const paci_shapes& s = h->s;
  const Layout& L = h->L;
  const int T = (int)L.T, d = s.d_model;
  if (s.kind == PACI_FIRST) {
    TRY(run(h, F_EMBED, (double)T * d * (8 + h->esz), [&] {
      return paci::embed_fwd(h->dt, ids, h->th(h->p.wte), h->th(h->p.wpe), A + L.blk[0].x, s.micro_batch, s.seq, d,
                             s.vocab, h->st);
    }));
    if (L.dropout) TRY(dropout(h, A + L.blk[0].x, nullptr, A + L.blk[0].x, h->drop(mb, 0, SITE_EMBED)));
    return blocks_fwd(h, A, A + L.blk[0].x, nullptr, out, mb);
  }
  if (s.kind == PACI_MIDDLE) return blocks_fwd(h, A, in, x0_copy, out, mb);
  TRY(blocks_fwd(h, A, in, x0_copy, A + L.s_y, mb));
  float* meanf = reinterpret_cast<float*>(A + L.s_meanf);
  float* rstdf = reinterpret_cast<float*>(A + L.s_rstdf);
  TRY(ln_fwd(h, A + L.s_y, A + L.s_nf, meanf, rstdf, h->p.lnf_g, h->p.lnf_b, nullptr));
  if (L.fused_head) {
    // logits reduced to (max, sum) per 64 columns inside the product, then per row
    paci::GemmArgs a{A + L.s_nf, d, h->W(h->p.w_lm), d, T, s.vocab, d, nullptr, 0, nullptr, nullptr, 0, nullptr,
                     h->arena + L.zeros};
    a.row_tgt = tgt;
    a.ce_part = reinterpret_cast<float*>(h->ws(L.w_cepart));
    a.ld_part = L.ngroups;
    a.ce_zt = reinterpret_cast<float*>(h->ws(L.w_zt));
    TRY(run(h, F_GEMM_FWD, 2.0 * T * s.vocab * d,
            [&] { return paci::gemm(h->dt, true, paci::GEMM_NT, paci::EPI_CE_STATS, a, 1, h->st); }));
    return run(h, F_CE, 8.0 * T * L.ngroups + 16.0 * T, [&] {
      return paci::ce_combine(a.ce_part, L.ngroups, L.ngroups, a.ce_zt, tgt, s.vocab,
                              reinterpret_cast<float*>(A + L.s_lse_ce), reinterpret_cast<float*>(out),
                              reinterpret_cast<float*>(h->ws(L.w_part)), T, h->st);
    });
  }
  float* z = reinterpret_cast<float*>(A + L.s_z);
  paci::GemmArgs a{A + L.s_nf, d, h->W(h->p.w_lm), d, T, s.vocab, d, z, L.ldz, nullptr, nullptr, 0, nullptr,
                   h->arena + L.zeros};
  TRY(run(h, F_GEMM_FWD, 2.0 * T * s.vocab * d,
          [&] { return paci::gemm(h->dt, true, paci::GEMM_NT, paci::EPI_STORE, a, 1, h->st); }));
  return run(h, F_CE, 4.0 * T * s.vocab, [&] {
    return paci::ce_fwd(z, L.ldz, tgt, reinterpret_cast<float*>(A + L.s_lse_ce), reinterpret_cast<float*>(out),
                        reinterpret_cast<float*>(h->ws(L.w_part)), T, s.vocab, h->st);
  });
}

}  // namespace

// ============================================================================================
// C ABI
// ============================================================================================
extern "C" int paci_param_count(const paci_shapes* s, int* n_tensors, int64_t* n_elements) {
  if (!s) return PACI_E_INVAL;
  const int v = validate_shapes(s, 1, 0);
  if (v) return v;
  const ParamTable p = build_params(*s);
  if (n_tensors) *n_tensors = (int)p.t.size();
  if (n_elements) *n_elements = p.total;
  return PACI_OK;
}

extern "C" int paci_param_info_at(const paci_shapes* s, int index, paci_param_info* out) {
  if (!s || !out) return PACI_E_INVAL;
  const int v = validate_shapes(s, 1, 0);
  if (v) return v;
  const ParamTable p = build_params(*s);
  if (index < 0 || index >= (int)p.t.size()) return PACI_E_INVAL;
  const TensorRef& t = p.t[index];
  memcpy(out->name, t.name, sizeof(out->name));
  out->rows = t.rows;
  out->cols = t.cols;
  out->offset = t.off;
  out->numel = t.numel;
  out->decay = t.decay ? 1 : 0;
  return PACI_OK;
}

extern "C" int paci_stage_arena_bytes(const paci_shapes* s, int K, int delay, size_t* bytes) {
  if (!bytes) return PACI_E_INVAL;
  const int v = validate_shapes(s, K, delay);
  if (v) return v;
  const ParamTable p = build_params(*s);
  *bytes = make_layout(*s, K, delay, p).total;
  return PACI_OK;
}

extern "C" int paci_stage_init(const paci_shapes* s, int K, int delay, void* dev_arena, size_t arena_bytes,
                               void* hip_stream, paci_stage** out) {
  if (!out || !dev_arena) return PACI_E_INVAL;
  if (reinterpret_cast<uintptr_t>(dev_arena) & 255) return PACI_E_INVAL;
  const int v = validate_shapes(s, K, delay);
  if (v) return v;
  paci_stage* h = new (std::nothrow) paci_stage();
  if (!h) return PACI_E_NOMEM;
  h->s = *s;
  h->fsm = paci_fsm{K, delay, 0, 0, 0, 0, 0};
  h->st = reinterpret_cast<hipStream_t>(hip_stream);
  h->arena = reinterpret_cast<char*>(dev_arena);
  h->p = build_params(*s);
  h->L = make_layout(*s, K, delay, h->p);
  h->dt = s->dtype == PACI_BF16 ? paci::DT_BF16 : paci::DT_F32;
  h->esz = s->dtype == PACI_BF16 ? 2 : 4;
  if (arena_bytes < h->L.total) {
    delete h;
    return PACI_E_NOMEM;
  }
  h->pairs = reinterpret_cast<float*>(h->arena + h->L.w_D);
  {
    const hipError_t se = static_scratch(&h->static_pairs);   // the stage's GPU is the current one
    if (se != hipSuccess) {
      g_init_hip_error = (int)se;
      delete h;
      return PACI_E_HIP;
    }
  }
  if (h->p.total >= (int64_t)INT32_MAX) {
    delete h;
    return PACI_E_UNSUPPORTED;
  }
  // AdamW table (entries never cross a tensor boundary) and the guard's ranges
  const std::vector<int4> chunks = adamw_table(h->p, h->L.wT, h->L.wdefer);
  const std::vector<int2> granges = guard_table(h->p);
  h->g_lazy = h->L.wdefer;       // G starts zero either way
  h->guard_full = !h->L.wdefer;
  hipError_t e = hipMemsetAsync(h->arena, 0, h->L.stash, h->st);  // theta, G, m, v, bf16 copy
  if (e == hipSuccess && h->L.fused_head)   // dz columns V .. ldz-1 stay zero (the dgrad reads them)
    e = hipMemsetAsync(h->arena + h->L.w_dz, 0, (size_t)h->esz * h->L.T * h->L.ldz, h->st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(h->arena + h->L.chunks, chunks.data(), chunks.size() * sizeof(int4), hipMemcpyHostToDevice,
                       h->st);
  if (e == hipSuccess && !granges.empty())
    e = hipMemcpyAsync(h->arena + h->L.guard, granges.data(), granges.size() * sizeof(int2), hipMemcpyHostToDevice,
                       h->st);
  std::vector<paci::WgradProblem> tabs;
  if (h->L.wdefer) tabs = wgrad_tables(h);
  if (e == hipSuccess && !tabs.empty())
    e = hipMemcpyAsync(h->arena + h->L.wgroup, tabs.data(), tabs.size() * sizeof(paci::WgradProblem),
                       hipMemcpyHostToDevice, h->st);
  if (e == hipSuccess) e = hipStreamSynchronize(h->st);
  if (e != hipSuccess) {
    g_init_hip_error = (int)e;
    delete h;
    return PACI_E_HIP;
  }
  *out = h;
  return PACI_OK;
}

extern "C" int paci_stage_destroy(paci_stage* h) {
  if (!h) return PACI_E_INVAL;
  for (auto& p : h->pending) {
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  for (auto e : h->free_ev) (void)hipEventDestroy(e);
  delete h;
  return PACI_OK;
}

static float* state_ptr(paci_stage* h, int what) {
  switch (what) {
    case PACI_PARAMS: return h->theta();
    case PACI_GRADS: return h->G();
    case PACI_EXP_AVG: return h->m();
    case PACI_EXP_AVG_SQ: return h->v();
  }
  return nullptr;
}

extern "C" int paci_stage_load(paci_stage* h, int what, const float* src, int64_t n, int on_device) {
  if (!h || !src || n != h->p.total) return PACI_E_INVAL;
  if (h->broken) return PACI_E_HIP;
  float* dst = state_ptr(h, what);
  if (!dst) return PACI_E_INVAL;
  if (what == PACI_GRADS) {
    TRY(flush_window(h));   // pending products belong to the G being replaced
    // the loaded values are G as it stands: added to, and guarded in full at the next update
    TRY(run(h, F_ADAMW, 0.0, [&] { return paci::adamw_ctl(reinterpret_cast<int*>(h->arena + h->L.ctl), 0, h->st); }));
    h->g_lazy = false;
    h->guard_full = true;
  }
  hipError_t e = hipMemcpyAsync(dst, src, (size_t)n * 4, on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice,
                                h->st);
  if (e == hipSuccess && what == PACI_PARAMS && h->dt == paci::DT_BF16) {
    e = paci::f32_to_bf16(h->theta(), h->arena + h->L.theta16, n, h->st);
    if (e == hipSuccess && refresh_wT(h) != PACI_OK) e = (hipError_t)h->last_hip;
  }
  if (e == hipSuccess && !on_device) e = hipStreamSynchronize(h->st);
  if (e != hipSuccess) {
    h->last_hip = (int)e;
    return PACI_E_HIP;
  }
  return PACI_OK;
}

extern "C" int paci_stage_read(paci_stage* h, int what, float* dst, int64_t n, int on_device) {
  if (!h || !dst || n != h->p.total) return PACI_E_INVAL;
  if (h->broken) return PACI_E_HIP;
  const float* src = state_ptr(h, what);
  if (!src) return PACI_E_INVAL;
  if (what == PACI_GRADS) {
    TRY(flush_window(h));
    TRY(materialize_g(h));
  }
  hipError_t e = hipMemcpyAsync(dst, src, (size_t)n * 4, on_device ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost,
                                h->st);
  if (e == hipSuccess && !on_device) e = hipStreamSynchronize(h->st);
  if (e != hipSuccess) {
    h->last_hip = (int)e;
    return PACI_E_HIP;
  }
  return PACI_OK;
}

extern "C" int paci_stage_forward(paci_stage* h, int mb, const void* dev_in, const int32_t* dev_targets,
                                  void* dev_out, int* version) {
  if (!h || !dev_in || !dev_out) return PACI_E_INVAL;
  if (h->s.kind == PACI_LAST && !dev_targets) return PACI_E_INVAL;
  if (h->broken) return PACI_E_HIP;
  const int chk = fsm_check_forward(h->fsm, mb);
  if (chk) return chk;
  const paci_shapes& s = h->s;
  const Layout& L = h->L;
  const int T = (int)L.T;
  char* sl = h->slot(mb);
  char* A = h->acts(mb);
  // what a checkpointed stage keeps: the input (and ids / targets) in the slot
  void* x0 = L.recompute ? (void*)(sl + L.c_x) : (void*)(A + L.blk[0].x);
  int r = PACI_OK;
  if (s.kind == PACI_FIRST) {
    int32_t* ids = reinterpret_cast<int32_t*>(sl + (L.recompute ? L.c_ids : L.s_ids));
    r = run(h, F_COPY, 8.0 * T, [&] {
      return hipMemcpyAsync(ids, dev_in, 4 * (size_t)T, hipMemcpyDeviceToDevice, h->st);
    });
    if (!r) r = stage_forward_into(h, A, nullptr, nullptr, ids, nullptr, dev_out, mb);
  } else if (s.kind == PACI_MIDDLE) {
    r = stage_forward_into(h, A, dev_in, x0, nullptr, nullptr, dev_out, mb);
  } else {
    int32_t* tgt = reinterpret_cast<int32_t*>(sl + (L.recompute ? L.c_tgt : L.s_tgt));
    r = run(h, F_COPY, 8.0 * T, [&] {
      return hipMemcpyAsync(tgt, dev_targets, 4 * (size_t)T, hipMemcpyDeviceToDevice, h->st);
    });
    if (!r) r = stage_forward_into(h, A, dev_in, x0, nullptr, tgt, dev_out, mb);
  }
  if (r) return r;
  const int t = fsm_commit_forward(h->fsm);
  if (version) *version = t;
  return PACI_OK;
}

static int stage_backward(paci_stage* h, int mb, const void* dev_grad_out, void* dev_grad_in, int* version) {
  if (!h) return PACI_E_INVAL;
  const paci_shapes& s = h->s;
  if (s.kind == PACI_LAST ? (dev_grad_out != nullptr) : (dev_grad_out == nullptr)) return PACI_E_INVAL;
  if (s.kind == PACI_FIRST && dev_grad_in) return PACI_E_INVAL;
  if (h->broken) return PACI_E_HIP;
  const int chk = fsm_check_backward(h->fsm, mb);
  if (chk) return chk;
  const Layout& L = h->L;
  const int T = (int)L.T, d = s.d_model;
  char* sl = h->slot(mb);
  char* A = h->acts(mb);   // the activations the backward differentiates
  const int32_t* ids = reinterpret_cast<const int32_t*>(sl + (L.recompute ? L.c_ids : L.s_ids));
  const int32_t* tgt = reinterpret_cast<const int32_t*>(sl + (L.recompute ? L.c_tgt : L.s_tgt));
  char* bufA = h->ws(L.w_dyA);
  char* bufB = h->ws(L.w_dyB);
  const void* dy = dev_grad_out;
  const int j = L.window ? h->fsm.c : 0;   // position in the window buffers
  const bool win = L.window || L.wdefer;
  // windowed: every block's output gradient lives in the window buffer
  char* dy_last = win ? h->win(L.win[s.n_layers - 1].dy, j, d) : bufA;
  int r = PACI_OK;
  if (L.recompute) {
    // checkpointed: the activations again, from the stored input, under the
    // parameters current now (the output, or loss, is discarded)
    void* out = s.kind == PACI_LAST ? (void*)h->ws(L.w_loss) : (void*)bufB;
    r = s.kind == PACI_FIRST ? stage_forward_into(h, A, nullptr, nullptr, ids, nullptr, out, mb)
                             : stage_forward_into(h, A, sl + L.c_x, A + L.blk[0].x, nullptr, tgt, out, mb);
  }
  if (!r && s.kind == PACI_LAST) {
    char* dz = h->ws(L.w_dz);
    char* dnf = h->ws(L.w_dnf);
    const float scale = 1.0f / ((float)T * (float)h->fsm.K);
    if (L.fused_head) {
      // the logits again (the parameters are those of the forward), into dL/dz
      paci::GemmArgs a{A + L.s_nf, d, h->W(h->p.w_lm), d, T, s.vocab, d, dz, L.ldz, nullptr, nullptr, 0, nullptr,
                       h->arena + L.zeros};
      a.row_tgt = tgt;
      a.row_lse = reinterpret_cast<const float*>(A + L.s_lse_ce);
      a.alpha = scale;
      r = run(h, F_GEMM_FWD, 2.0 * T * s.vocab * d,
              [&] { return paci::gemm(h->dt, false, paci::GEMM_NT, paci::EPI_CE_GRAD, a, 1, h->st); });
    } else {
      const float* z = reinterpret_cast<const float*>(A + L.s_z);
      r = run(h, F_CE, (double)T * L.ldz * (4 + h->esz), [&] {
        return paci::ce_bwd(h->dt, z, L.ldz, tgt, reinterpret_cast<const float*>(A + L.s_lse_ce), dz, T, s.vocab,
                            scale, h->st);
      });
    }
    if (!r) r = linear_wgrad(h, dz, L.ldz, A + L.s_nf, d, s.vocab, d, T, h->p.w_lm);
    if (!r) r = linear_dgrad(h, dz, L.ldz, h->p.w_lm, T, d, s.vocab, paci::EPI_STORE, dnf, nullptr, -1, false);
    if (!r)   // the last block's output gradient; G_b2 of that block += its column sums
      r = ln_bwd(h, dnf, A + L.s_y, reinterpret_cast<const float*>(A + L.s_meanf),
                 reinterpret_cast<const float*>(A + L.s_rstdf), h->p.lnf_g, h->p.lnf_b, nullptr, dy_last,
                 L.dropout ? -1 : h->p.blocks[s.n_layers - 1].b_2);
    dy = dy_last;
  } else if (!r && win) {
    r = run(h, F_COPY, 2.0 * act_bytes(h), [&] {
      return hipMemcpyAsync(dy_last, dev_grad_out, act_bytes(h), hipMemcpyDeviceToDevice, h->st);
    });
    dy = dy_last;
  }
  for (int l = s.n_layers - 1; l >= 0 && !r; --l) {
    void* dx;
    if (l == 0 && s.kind != PACI_FIRST && dev_grad_in)
      dx = dev_grad_in;
    else if (l > 0 && win)
      dx = h->win(L.win[l - 1].dy, j, d);
    else
      dx = (dy == bufA) ? bufB : bufA;
    // every block's dy but the given stage output gradient came out of a LayerNorm backward
    r = block_bwd(h, A, l, dy, dx, l < s.n_layers - 1 || s.kind == PACI_LAST, j, mb);
    dy = dx;
  }
  if (!r && L.wdefer) {
    int* ctl = reinterpret_cast<int*>(h->arena + L.ctl);
    r = wgrad_grouped(h, L.recompute ? 0 : mb % L.n_slots, h->g_lazy, h->fsm.c + 1 == h->fsm.K ? ctl : nullptr);
    if (!r) h->g_lazy = false;
  }
  if (!r && s.kind == PACI_FIRST && L.dropout) {   // through the embedding dropout
    r = dropout(h, dy, nullptr, h->ws(L.w_g2), h->drop(mb, 0, SITE_EMBED));
    dy = h->ws(L.w_g2);
  }
  if (!r && s.kind == PACI_FIRST) {
    r = run(h, F_EMBED, (double)T * d * (h->esz + 8), [&] {
      return paci::embed_bwd(h->dt, ids, dy, h->g(h->p.wte),
                             h->g(h->p.wpe), s.micro_batch, s.seq, d, s.vocab, h->st);
    });
  }
  if (r) return r;
  const int t = fsm_commit_backward(h->fsm);
  if (version) *version = t;
  return h->fsm.c == h->fsm.K ? PACI_STEP_DUE : PACI_OK;
}

extern "C" int paci_stage_backward(paci_stage* h, int mb, const void* dev_grad_out, void* dev_grad_in,
                                   int* version) {
  return stage_backward(h, mb, dev_grad_out, dev_grad_in, version);
}

extern "C" int paci_stage_backward_static(paci_stage* h, int mb, const void* dev_grad_out, void* dev_grad_in,
                                          int* version) {
  if (!h) return PACI_E_INVAL;
  const size_t need = 4 * (size_t)paci::attn_bwd_workspace_floats(h->dt, h->s.micro_batch, h->s.seq, h->s.n_heads);
  if (need > kStaticScratchBytes) return PACI_E_SCRATCH;
  if (h->static_pairs == nullptr) return PACI_E_HIP;
  float* own = h->pairs;
  h->pairs = reinterpret_cast<float*>(h->static_pairs);   // every entry is rewritten by the call
  h->no_events = true;
  const int r = stage_backward(h, mb, dev_grad_out, dev_grad_in, version);
  h->pairs = own;
  h->no_events = false;
  return r;
}

extern "C" int paci_stage_step(paci_stage* h, int* new_version) {
  if (!h) return PACI_E_INVAL;
  if (h->fsm.c != h->fsm.K) return PACI_E_NOT_DUE;
  if (h->broken) return PACI_E_HIP;
  const paci_shapes& s = h->s;
  paci::AdamwArgs a;
  a.lr = s.lr;
  a.beta1 = s.beta1;
  a.beta2 = s.beta2;
  a.eps = s.eps;
  a.weight_decay = s.weight_decay;
  a.lr_min_ratio = s.lr_min_ratio;
  a.lr_warmup = s.lr_warmup;
  a.lr_total = s.lr_total;
  int* ctl = reinterpret_cast<int*>(h->arena + h->L.ctl);
  TRY(flush_window(h));
  // the non-finite guard decides on the device: no host synchronization. The
  // window's last backward already checked the block matrices' G as it wrote
  // them (grouped weight gradients); the guard reads the rest, or all of G.
  if (h->guard_full) {
    TRY(run(h, F_ADAMW, 4.0 * (double)h->p.total, [&] { return paci::adamw_guard(h->G(), h->p.total, ctl, h->st); }));
  } else {
    double n = 0;
    for (const auto& t : h->p.t)
      if (!is_block_matrix(h->p, t.off)) n += (double)t.numel;
    TRY(run(h, F_ADAMW, 4.0 * n, [&] {
      return paci::adamw_guard_ranges(h->G(), reinterpret_cast<const int2*>(h->arena + h->L.guard), h->L.nguard, ctl,
                                      h->st);
    }));
  }
  const int r = run(h, F_ADAMW, 30.0 * (double)h->p.total, [&] {
    return paci::adamw(h->theta(), h->G(), h->m(), h->v(),
                       h->dt == paci::DT_BF16 ? (void*)(h->arena + h->L.theta16) : nullptr,
                       h->L.wT ? (void*)(h->arena + h->L.theta16T) : nullptr,
                       reinterpret_cast<const int4*>(h->arena + h->L.chunks), h->L.nchunks, a, ctl, h->st);
  });
  if (r) return r;
  // counts the update as applied or skipped and clears the flag for the next window
  TRY(run(h, F_ADAMW, 0.0, [&] { return paci::adamw_ctl(ctl, 1, h->st); }));
  h->g_lazy = h->L.wdefer;
  h->guard_full = !h->L.wdefer;
  fsm_commit_step(h->fsm);
  h->win_done = 0;
  if (new_version) *new_version = h->fsm.t;
  return PACI_OK;
}

extern "C" int paci_stage_run_events(paci_stage* h, int n, const int32_t* kinds, const int32_t* idx,
                                     const void* dev_in_all, const int32_t* dev_targets_all,
                                     const void* dev_grad_out_all, void* dev_out_all, void* dev_grad_in_all,
                                     int32_t* host_stamps) {
  if (!h || n < 0 || !dev_in_all || (n > 0 && (!kinds || !idx))) return PACI_E_INVAL;
  for (int e = 0; e < n; ++e)   // the whole list is checked before any event runs
    if (kinds[e] < 0 || kinds[e] > 2 || (kinds[e] < 2 && idx[e] < 0)) return PACI_E_INVAL;
  const paci_shapes& s = h->s;
  if (s.kind == PACI_LAST && !dev_targets_all) return PACI_E_INVAL;
  if (s.kind != PACI_LAST && !dev_grad_out_all) return PACI_E_INVAL;
  const int64_t T = h->L.T;
  const size_t act = act_bytes(h);
  const size_t in_stride = s.kind == PACI_FIRST ? 4 * (size_t)T : act;
  const size_t out_stride = s.kind == PACI_LAST ? sizeof(float) : act;
  // scratch outputs when the caller discards them
  char* out_scratch = h->ws(h->L.w_dyB);
  float* loss_scratch = reinterpret_cast<float*>(h->ws(h->L.w_loss));
  int r = PACI_OK;
  for (int e = 0; e < n; ++e) {
    const int i = idx[e];
    int ver = 0;
    if (kinds[e] == 0) {
      const char* in = reinterpret_cast<const char*>(dev_in_all) + in_stride * i;
      const int32_t* tg = dev_targets_all ? dev_targets_all + T * i : nullptr;
      void* out = dev_out_all ? (void*)(reinterpret_cast<char*>(dev_out_all) + out_stride * i)
                              : (s.kind == PACI_LAST ? (void*)loss_scratch : (void*)out_scratch);
      // a middle/first stage writes its output before any backward reads the scratch buffer
      r = paci_stage_forward(h, i, in, tg, out, &ver);
      if (r < 0) return r;
      if (host_stamps) host_stamps[3 * i] = ver;
    } else if (kinds[e] == 1) {
      const void* go = s.kind == PACI_LAST ? nullptr
                                           : (const void*)(reinterpret_cast<const char*>(dev_grad_out_all) + act * i);
      void* gi = (s.kind != PACI_FIRST && dev_grad_in_all) ? (void*)(reinterpret_cast<char*>(dev_grad_in_all) + act * i)
                                                           : nullptr;
      r = paci_stage_backward(h, i, go, gi, &ver);
      if (r < 0) return r;
      if (host_stamps) {
        host_stamps[3 * i + 1] = ver;
        host_stamps[3 * i + 2] = ver - host_stamps[3 * i];
      }
    } else {
      r = paci_stage_step(h, &ver);
      if (r < 0) return r;
    }
  }
  return PACI_OK;
}

extern "C" int paci_stage_run(paci_stage* h, int M, const void* dev_in_all, const int32_t* dev_targets_all,
                              const void* dev_grad_out_all, void* dev_out_all, void* dev_grad_in_all,
                              int32_t* host_stamps) {
  if (!h || M < 0) return PACI_E_INVAL;
  if (h->fsm.next_f != 0 || h->fsm.next_b != 0 || h->fsm.c != 0) return PACI_E_ORDER;   // a fresh replay
  std::vector<int32_t> kinds(2 * (size_t)M + M / h->fsm.K + 1), idx(kinds.size());
  int n = 0;
  const int r = paci_schedule(M, h->fsm.K, h->fsm.delay, kinds.data(), idx.data(), (int)kinds.size(), &n);
  if (r) return r;
  return paci_stage_run_events(h, n, kinds.data(), idx.data(), dev_in_all, dev_targets_all, dev_grad_out_all,
                               dev_out_all, dev_grad_in_all, host_stamps);
}

extern "C" int paci_stage_updates(paci_stage* h, int32_t* applied, int32_t* skipped) {
  if (!h || !applied || !skipped) return PACI_E_INVAL;
  if (h->broken) return PACI_E_HIP;
  int ctl[4] = {0, 0, 0, 0};
  hipError_t e = hipMemcpyAsync(ctl, h->arena + h->L.ctl, sizeof(ctl), hipMemcpyDeviceToHost, h->st);
  if (e == hipSuccess) e = hipStreamSynchronize(h->st);
  if (e != hipSuccess) {
    h->last_hip = (int)e;
    return PACI_E_HIP;
  }
  *applied = ctl[1];
  *skipped = ctl[2];
  return PACI_OK;
}

extern "C" int paci_stage_resume(paci_stage* h, int32_t version, int32_t next_mb, int32_t applied,
                                 int32_t skipped) {
  if (!h || version < 0 || next_mb < 0 || applied < 0 || skipped < 0) return PACI_E_INVAL;
  if (h->broken) return PACI_E_HIP;
  if (h->fsm.q != 0 || h->fsm.c != 0 || h->fsm.next_f != h->fsm.next_b) return PACI_E_ORDER;   // drained only
  const int ctl[4] = {0, applied, skipped, 0};
  hipError_t e = hipMemcpyAsync(h->arena + h->L.ctl, ctl, sizeof(ctl), hipMemcpyHostToDevice, h->st);
  if (e == hipSuccess) e = hipStreamSynchronize(h->st);
  if (e != hipSuccess) {
    h->last_hip = (int)e;
    return PACI_E_HIP;
  }
  h->fsm.t = version;
  h->fsm.next_f = h->fsm.next_b = next_mb;
  h->win_done = 0;
  return PACI_OK;
}

extern "C" int paci_stage_reset_counters(paci_stage* h) {
  if (!h) return PACI_E_INVAL;
  if (!h->broken) TRY(flush_window(h));   // G keeps what the backwards so far accumulated
  h->win_done = 0;
  if (!h->broken)   // update counts restart with the version (bias correction from step 1)
    TRY(run(h, F_ADAMW, 0.0, [&] { return paci::adamw_ctl(reinterpret_cast<int*>(h->arena + h->L.ctl), 2, h->st); }));
  h->fsm.t = h->fsm.c = h->fsm.q = h->fsm.next_f = h->fsm.next_b = 0;
  return PACI_OK;
}

extern "C" int paci_stage_counters(const paci_stage* h, paci_counters* out) {
  if (!h || !out) return PACI_E_INVAL;
  fsm_counters(h->fsm, out);
  return PACI_OK;
}

extern "C" int paci_stage_sync(paci_stage* h) {
  if (!h) return PACI_E_INVAL;
  const hipError_t e = hipStreamSynchronize(h->st);
  if (e != hipSuccess) {
    h->last_hip = (int)e;
    return PACI_E_HIP;
  }
  return PACI_OK;
}

extern "C" int paci_last_hip_error(const paci_stage* h) { return h ? h->last_hip : g_init_hip_error; }

extern "C" const char* paci_strerror(int status) {
  switch (status) {
    case PACI_OK: return "ok";
    case PACI_STEP_DUE: return "optimizer step due";
    case PACI_E_INVAL: return "invalid argument";
    case PACI_E_UNSUPPORTED: return "unsupported shape or dtype";
    case PACI_E_NOMEM: return "arena too small";
    case PACI_E_ORDER: return "micro-batch out of order";
    case PACI_E_BACKPRESSURE: return "forward refused by the admission rule (q > delay)";
    case PACI_E_STEP_PENDING: return "optimizer step pending";
    case PACI_E_NOT_DUE: return "optimizer step not due";
    case PACI_E_HIP: return "HIP runtime error";
    case PACI_E_SCRATCH: return "the call's scratch exceeds the library's static scratch buffer";
  }
  return "unknown status";
}

extern "C" int paci_kernel_family_count(void) { return F_COUNT; }
extern "C" const char* paci_kernel_family_name(int family) {
  return (family >= 0 && family < F_COUNT) ? kFamilyNames[family] : nullptr;
}

extern "C" int paci_stage_set_timing(paci_stage* h, int enable) {
  if (!h) return PACI_E_INVAL;
  if (!enable && h->timing) {
    const hipError_t e = hipStreamSynchronize(h->st);
    drain_timing(h);
    if (e != hipSuccess) {
      h->last_hip = (int)e;
      h->timing = false;
      return PACI_E_HIP;
    }
  }
  if (enable && !h->timing) {
    for (int i = 0; i < F_COUNT; ++i) {
      h->launches[i] = 0;
      h->ms[i] = h->work[i] = 0;
    }
  }
  h->timing = enable != 0;
  return PACI_OK;
}

extern "C" int paci_stage_kernel_times(paci_stage* h, int family, int64_t* launches, double* ms, double* work) {
  if (!h || family < 0 || family >= F_COUNT) return PACI_E_INVAL;
  drain_timing(h);
  if (launches) *launches = h->launches[family];
  if (ms) *ms = h->ms[family];
  if (work) *work = h->work[family];
  return PACI_OK;
}
