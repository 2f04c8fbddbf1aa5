// Host runtime and C ABI of the dllm library (see include/dllm.h).
//
// The runtime validates arguments, carves the caller's workspace into the
// step's buffers, evaluates the threshold schedule on the host in float64, and
// enqueues the kernels of one step on the caller's stream:
//   embed -> n_layers x [norm, qkv+rope, attention, o-proj+residual, norm,
//   gate/up+swiglu, down+residual] -> final norm of the block rows -> fused LM
//   head + vocabulary reduction -> commit.
// dllm_generate runs the semi-autoregressive block loop (Section 4.3) and
// waits once per step for the block-finished flag, which the commit kernel
// publishes to a coherent pinned host word the host polls.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <mutex>

#include <string>
#include <vector>

#include "../../include/dllm.h"

#include "kernels.h"

using namespace dllm;

namespace {

thread_local std::string g_last_error;

struct ApiError {
  int code;
  std::string msg;
};

[[noreturn]] void fail(int code, const std::string& msg) { throw ApiError{code, msg}; }
void require(bool ok, int code, const std::string& msg) {
  if (!ok) fail(code, msg);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

struct ProfEvent {
  int kind;
  hipEvent_t start, stop;
};

struct dllm_model {
  dllm_model_cfg cfg;
  std::vector<const void*> w;
  bf16_t* head_tiled = nullptr;  // bf16: tiled copy of the LM head, in the caller's model buffer
  // bf16, after dllm_model_pack_weights: packed copies of every layer's q/k/v,
  // output, gate/up and down weights (in the caller's buffer; offsets per layer)
  bf16_t* packed = nullptr;
  std::vector<size_t> packed_off;  // [layer * 4 + {0: qkv, 1: o, 2: gate/up, 3: down}] in elements
  // coherent pinned word the commit kernel publishes each step's done/error
  // word to (tagged with the step's sequence number), and its device address
  int32_t* step_flag = nullptr;
  int32_t* step_flag_dev = nullptr;
  int step_seq = 0;
  uint32_t prof_mask = 0;  // bit k: record launches of kind k
  int prof_every = 1;      // record one launch in prof_every of each kind
  int64_t prof_seen[8] = {};
  std::vector<ProfEvent> events;
  size_t n_events = 0;
};

namespace {

// ---------------------------------------------------------------- layout
struct Layout {
  size_t h, a_attn, q, k, vt, attn, a_mlp, u, hb, cosb, sinb;
  size_t raw, gate, up, logits;                  // fp32 path
  size_t part_m, part_s, part_i, ticket, hbf;    // bf16 head
  size_t splitk;                                 // bf16 split-K GEMM partials
  size_t attn_part, attn_ticket;                 // bf16 key-split attention states and tickets
  size_t conf, argmax, all_done, err;            // step scratch
  size_t total;
};

// Buffers whose contents outlive a call (the residual h, the RoPE tables, the
// error word) and everything sized by B and L alone come first, so their
// offsets do not depend on `rows`: calls on one workspace with different row
// counts (dllm_layer, then dllm_head) see the same h and tables.  The buffers
// sized by the head rows follow.
Layout make_layout(const dllm_model_cfg& c, int B, int L, int rows) {
  const size_t M = (size_t)B * L, d = c.d_model, F = c.d_ff, hd = c.head_dim;
  const size_t act = c.dtype == DLLM_F32 ? 4 : 2;
  const size_t R = (size_t)B * rows;
  Layout o{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  o.h = take(M * d * 4);
  o.a_attn = take(M * d * act);
  o.q = take(M * c.n_heads * hd * act);
  o.k = take(M * c.n_kv_heads * hd * act);
  o.vt = take(M * c.n_kv_heads * hd * act);     // fp32, or IEEE half for bf16 models
  o.attn = take(M * c.n_heads * hd * act);
  o.a_mlp = take(M * d * act);
  o.u = take(M * F * act);
  o.cosb = take((size_t)L * hd / 2 * 4);
  o.sinb = take((size_t)L * hd / 2 * 4);
  o.all_done = take(4);
  o.err = take(4);
  if (c.dtype == DLLM_F32) {
    o.raw = take(M * (c.n_heads + 2 * c.n_kv_heads) * hd * 4);
    o.gate = take(M * F * 4);
    o.up = take(M * F * 4);
  } else {
    o.ticket = take(4);
    o.hbf = take((size_t)HEAD_FRAG_ROWS * d * 2);
    o.attn_ticket = take((size_t)B * c.n_heads * 4);
    o.attn_part = take(attn_split_bytes(B, c.n_heads));
  }
  // sized by the head rows
  o.hb = take(R * d * act);
  o.conf = take(R * 4);
  o.argmax = take(R * 4);
  if (c.dtype == DLLM_F32) {
    o.logits = take(R * c.vocab * 4);
  } else {
    const size_t tiles = head_bf16_tiles(c.vocab);
    o.part_m = take(tiles * R * 4);
    o.part_s = take(tiles * R * 4);
    o.part_i = take(tiles * R * 4);
    // split-K partials of the full forward (B L rows) and of a cached step's
    // forward (B rows rows); nothing in them outlives a call
    const int qkv_n = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
    size_t sk = 0;
    for (const int mm : {(int)M, (int)R}) {
      if (mm == 0) continue;
      sk = std::max({sk, gemm_bf16_splitk_bytes(mm, qkv_n, c.d_model, EPI_QKV_ROPE),
                     gemm_bf16_splitk_bytes(mm, c.d_model, c.n_heads * c.head_dim, EPI_RESID),
                     gemm_bf16_splitk_bytes(mm, 2 * c.d_ff, c.d_model, EPI_SWIGLU),
                     gemm_bf16_splitk_bytes(mm, c.d_model, c.d_ff, EPI_RESID)});
    }
    o.splitk = take(sk);
  }
  o.total = off;
  return o;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

void check_model(const dllm_model* m) { require(m != nullptr, DLLM_EINVAL, "model is NULL"); }

void check_ws(const dllm_model* m, int B, int L, int rows, void* ws, size_t bytes, Layout* lay) {
  require(B >= 1 && B <= 16, DLLM_EUNSUPPORTED, "batch must be in [1, 16]");
  require(L >= 1, DLLM_ESHAPE, "sequence length must be >= 1");
  require(rows >= 0 && rows <= L, DLLM_ESHAPE, "rows out of range");
  if (m->cfg.dtype == DLLM_BF16)
    require((long)B * rows <= head_bf16_max_rows(), DLLM_EUNSUPPORTED, "B * rows exceeds the LM-head kernel limit");
  else
    require(L <= 8000, DLLM_EUNSUPPORTED, "float32 attention keeps all scores in LDS: L <= 8000");
  require(ws != nullptr, DLLM_EINVAL, "workspace is NULL");
  require(((uintptr_t)ws & 255) == 0, DLLM_EINVAL, "workspace must be 256-byte aligned");
  *lay = make_layout(m->cfg, B, L, rows);
  require(bytes >= lay->total, DLLM_ENOMEM, "workspace too small: need " + std::to_string(lay->total) + " bytes");
}

// ---------------------------------------------------------------- profiling
struct ProfScope {
  dllm_model* m;
  hipStream_t s;
  ProfEvent* ev = nullptr;
  ProfScope(const dllm_model* mc, int kind, hipStream_t st) : m(const_cast<dllm_model*>(mc)), s(st) {
    if (!(m->prof_mask & (1u << kind))) return;
    if (m->prof_seen[kind]++ % m->prof_every != 0) return;
    if (m->n_events == m->events.size()) {
      ProfEvent e{};
      hip_check(hipEventCreate(&e.start), "hipEventCreate");
      hip_check(hipEventCreate(&e.stop), "hipEventCreate");
      m->events.push_back(e);
    }
    ev = &m->events[m->n_events++];
    ev->kind = kind;
    hip_check(hipEventRecord(ev->start, s), "hipEventRecord");
  }
  ~ProfScope() {
    if (ev) (void)hipEventRecord(ev->stop, s);
  }
};

enum { PK_QKV = 0, PK_ATTN = 1, PK_HEAD = 2, PK_COMMIT = 3, PK_NORM = 4, PK_GATEUP = 5, PK_OPROJ = 6, PK_DOWN = 7 };

const void* W(const dllm_model* m, int i) { return m->w[i]; }
const bf16_t* Wb(const dllm_model* m, int i) { return static_cast<const bf16_t*>(m->w[i]); }
const float* Wf(const dllm_model* m, int i) { return static_cast<const float*>(m->w[i]); }

// ---------------------------------------------------------------- key/value cache
// Per layer l: keys [B, Hkv, L, hd] (after RoPE) at l * 2 * S and values^T
// [B, Hkv, hd, L] at l * 2 * S + S, S = the 256-byte-rounded size of one of
// them (float32 for an fp32 model, bf16 keys and IEEE-half values for bf16).
size_t kv_slab_bytes(const dllm_model_cfg& c, int B, int L) {
  return align256((size_t)B * c.n_kv_heads * L * c.head_dim * (c.dtype == DLLM_F32 ? 4 : 2));
}
size_t kv_cache_bytes(const dllm_model_cfg& c, int B, int L) { return 2 * kv_slab_bytes(c, B, L) * c.n_layers; }

// Rows of the sequences a layer works on, and where its keys/values go: a
// full forward has Lq = L, pos0 = 0 and keeps them in the workspace (k, vt
// null) or stores them in the cache; a cached step has the block's Lq rows at
// positions pos0 .. pos0 + Lq - 1 and attends over the cache.
struct LayerRows {
  int Lq, pos0;
  void* k;
  void* vt;
};

LayerRows cache_rows(const dllm_model* m, void* kv, int layer, int B, int L, int Lq, int pos0) {
  const size_t S = kv_slab_bytes(m->cfg, B, L);
  char* base = static_cast<char*>(kv) + (size_t)layer * 2 * S;
  return LayerRows{Lq, pos0, base, base + S};
}

void check_kv(const dllm_model* m, int B, int L, const void* kv, size_t bytes) {
  require(kv != nullptr, DLLM_EINVAL, "kv_cache is NULL");
  require(((uintptr_t)kv & 255) == 0, DLLM_EINVAL, "kv_cache must be 256-byte aligned");
  const size_t need = kv_cache_bytes(m->cfg, B, L);
  require(bytes >= need, DLLM_ENOMEM, "kv_cache too small: need " + std::to_string(need) + " bytes");
}

// ---------------------------------------------------------------- forward pieces
// h[b rows + i] = embedding of x[b, row0 + i] (rows = L, row0 = 0: every
// position); with rope set, first the RoPE tables for all L positions, which
// also clears the error word (a decode builds them once, before its first
// step, after clearing the word in the state initialisation; each commit
// clears it after reporting).
void run_embed(const dllm_model* m, const int32_t* x, int B, int L, int row0, int rows, void* ws, const Layout& lay,
               hipStream_t s, bool rope = true) {
  const auto& c = m->cfg;
  if (rope)
    launch_rope_table(at<float>(ws, lay.cosb), at<float>(ws, lay.sinb), L, c.head_dim, c.rope_base,
                      at<int>(ws, lay.err), s);
  const bool bf = c.dtype == DLLM_BF16;
  launch_embed(x, W(m, 0), c.dtype, at<float>(ws, lay.h), B, rows, L, row0, c.d_model, c.vocab, at<int>(ws, lay.err),
               s, bf ? at<int>(ws, lay.attn_ticket) : nullptr, bf ? B * c.n_heads : 0);
}

void gemm_bf16(const dllm_model* m, GemmArgs g, void* ws, const Layout& lay, hipStream_t s, int kind,
               PendingResid* defer = nullptr) {
  g.splitk_buf = at<float>(ws, lay.splitk);
  ProfScope p(m, kind, s);
  launch_gemm_bf16(g, s, defer);
}

// RMSNorm of every row of h into out; split-K partials still pending from the
// previous residual GEMM (pend non-null with split > 0) are added to h first,
// in the same pass, and then cleared.
void norm_rows_bf16(const dllm_model* m, float* h, PendingResid* pend, const void* gain, void* out, int B, int L,
                    hipStream_t s) {
  const auto& c = m->cfg;
  ProfScope p(m, PK_NORM, s);
  if (pend && pend->split > 0) {
    launch_resid_rmsnorm(h, *pend, static_cast<const bf16_t*>(gain), static_cast<bf16_t*>(out), B * L, c.d_model,
                         c.rms_eps, s);
    *pend = PendingResid{};
  } else {
    launch_rmsnorm(h, gain, out, 1, B, L, L, 0, c.d_model, c.rms_eps, s);
  }
}

// The weight side of a layer's four GEMMs (q/k/v, output, gate/up, down).
GemmArgs layer_gemm(const dllm_model* m, int layer, int which) {
  const auto& c = m->cfg;
  const int base = 1 + 9 * layer, hd = c.head_dim;
  GemmArgs g{};
  switch (which) {
    case 0:
      g.epi = EPI_QKV_ROPE;
      g.N = (c.n_heads + 2 * c.n_kv_heads) * hd;
      g.K = c.d_model;
      g.W0 = Wb(m, base + 1);
      g.W1 = Wb(m, base + 2);
      g.W2 = Wb(m, base + 3);
      g.n0 = c.n_heads * hd;
      g.n1 = c.n_kv_heads * hd;
      break;
    case 1:
      g.epi = EPI_RESID;
      g.N = c.d_model;
      g.K = c.n_heads * hd;
      g.W0 = Wb(m, base + 4);
      g.n0 = c.d_model;
      break;
    case 2:
      g.epi = EPI_SWIGLU;
      g.N = 2 * c.d_ff;
      g.K = c.d_model;
      g.W0 = Wb(m, base + 6);
      g.W1 = Wb(m, base + 7);
      g.n0 = c.d_ff;
      g.n1 = c.d_ff;
      break;
    default:
      g.epi = EPI_RESID;
      g.N = c.d_model;
      g.K = c.d_ff;
      g.W0 = Wb(m, base + 8);
      g.n0 = c.d_model;
      break;
  }
  if (m->packed) g.Wp = m->packed + m->packed_off[(size_t)layer * 4 + which];
  return g;
}

// One layer (part 0: attention half, 1: MLP half, 2: both) on the B * Lq rows
// of h (rows: see LayerRows; null = the full sequence, keys/values in the
// workspace).  carry_in holds split-K partials the previous layer's down
// projection left pending (added by this layer's first norm); with carry_out
// non-null the down projection leaves its own partials there for the next
// layer instead of reducing them.  The output projection's partials are folded
// into the MLP norm when both halves run here.  Without carries h is complete
// when the call returns.
void run_layer_bf16(const dllm_model* m, int layer, int part, int B, int L, void* ws, const Layout& lay,
                    hipStream_t s, PendingResid* carry_in = nullptr, PendingResid* carry_out = nullptr,
                    const LayerRows* rows = nullptr) {
  const auto& c = m->cfg;
  const int base = 1 + 9 * layer;
  const int Lq = rows ? rows->Lq : L, pos0 = rows ? rows->pos0 : 0;
  const int M = B * Lq, d = c.d_model, hd = c.head_dim;
  float* h = at<float>(ws, lay.h);
  PendingResid mid;  // output-projection partials, consumed by the MLP norm
  if (part == 0 || part == 2) {
    norm_rows_bf16(m, h, carry_in, W(m, base + 0), at<void>(ws, lay.a_attn), B, Lq, s);
    GemmArgs g = layer_gemm(m, layer, 0);
    g.M = M;
    g.A = at<bf16_t>(ws, lay.a_attn);
    g.q = at<bf16_t>(ws, lay.q);
    g.k = rows && rows->k ? static_cast<bf16_t*>(rows->k) : at<bf16_t>(ws, lay.k);
    g.vt = rows && rows->vt ? static_cast<f16_t*>(rows->vt) : at<f16_t>(ws, lay.vt);
    g.cosb = at<float>(ws, lay.cosb);
    g.sinb = at<float>(ws, lay.sinb);
    g.B = B;
    g.L = L;
    g.Lq = Lq;
    g.pos0 = pos0;
    g.Hq = c.n_heads;
    g.Hkv = c.n_kv_heads;
    g.err = at<int>(ws, lay.err);
    gemm_bf16(m, g, ws, lay, s, PK_QKV);
    {
      ProfScope p(m, PK_ATTN, s);
      launch_attn_bf16(g.q, g.k, g.vt, at<bf16_t>(ws, lay.attn), B, Lq, L, c.n_heads, c.n_kv_heads, s,
                       at<float>(ws, lay.attn_part), at<int>(ws, lay.attn_ticket));
    }
    GemmArgs o = layer_gemm(m, layer, 1);
    o.M = M;
    o.A = at<bf16_t>(ws, lay.attn);
    o.resid = h;
    gemm_bf16(m, o, ws, lay, s, PK_OPROJ, part == 2 ? &mid : nullptr);
  }
  if (part == 1 || part == 2) {
    norm_rows_bf16(m, h, part == 1 ? carry_in : &mid, W(m, base + 5), at<void>(ws, lay.a_mlp), B, Lq, s);
    GemmArgs g = layer_gemm(m, layer, 2);
    g.M = M;
    g.A = at<bf16_t>(ws, lay.a_mlp);
    g.out = at<bf16_t>(ws, lay.u);
    gemm_bf16(m, g, ws, lay, s, PK_GATEUP);
    GemmArgs dn = layer_gemm(m, layer, 3);
    dn.M = M;
    dn.A = at<bf16_t>(ws, lay.u);
    dn.resid = h;
    gemm_bf16(m, dn, ws, lay, s, PK_DOWN, carry_out);
  }
}

void run_layer_f32(const dllm_model* m, int layer, int part, int B, int L, void* ws, const Layout& lay,
                   hipStream_t s, const LayerRows* rows = nullptr) {
  const auto& c = m->cfg;
  const int base = 1 + 9 * layer;
  const int Lq = rows ? rows->Lq : L, pos0 = rows ? rows->pos0 : 0;
  const int M = B * Lq, d = c.d_model, hd = c.head_dim, F = c.d_ff;
  float* kk = rows && rows->k ? static_cast<float*>(rows->k) : at<float>(ws, lay.k);
  float* vv = rows && rows->vt ? static_cast<float*>(rows->vt) : at<float>(ws, lay.vt);
  const int nq = c.n_heads * hd, nkv = c.n_kv_heads * hd, nraw = nq + 2 * nkv;
  float* h = at<float>(ws, lay.h);
  if (part == 0 || part == 2) {
    float* a = at<float>(ws, lay.a_attn);
    float* raw = at<float>(ws, lay.raw);
    {
      ProfScope p(m, PK_NORM, s);
      launch_rmsnorm(h, W(m, base + 0), a, 0, B, Lq, Lq, 0, d, c.rms_eps, s);
    }
    {
      ProfScope p(m, PK_QKV, s);
      launch_gemm_f32(a, Wf(m, base + 1), raw, M, nq, d, nraw, false, s);
      launch_gemm_f32(a, Wf(m, base + 2), raw + nq, M, nkv, d, nraw, false, s);
      launch_gemm_f32(a, Wf(m, base + 3), raw + nq + nkv, M, nkv, d, nraw, false, s);
    }
    launch_rope_split_f32(raw, at<float>(ws, lay.cosb), at<float>(ws, lay.sinb), at<float>(ws, lay.q), kk, vv, B,
                          Lq, L, pos0, c.n_heads, c.n_kv_heads, hd, s);
    {
      ProfScope p(m, PK_ATTN, s);
      launch_attn_f32(at<float>(ws, lay.q), kk, vv, at<float>(ws, lay.attn), B, Lq, L, c.n_heads, c.n_kv_heads, hd,
                      s);
    }
    ProfScope p(m, PK_OPROJ, s);
    launch_gemm_f32(at<float>(ws, lay.attn), Wf(m, base + 4), h, M, d, nq, d, true, s);
  }
  if (part == 1 || part == 2) {
    float* a = at<float>(ws, lay.a_mlp);
    {
      ProfScope p(m, PK_NORM, s);
      launch_rmsnorm(h, W(m, base + 5), a, 0, B, Lq, Lq, 0, d, c.rms_eps, s);
    }
    {
      ProfScope p(m, PK_GATEUP, s);
      launch_gemm_f32(a, Wf(m, base + 6), at<float>(ws, lay.gate), M, F, d, F, false, s);
      launch_gemm_f32(a, Wf(m, base + 7), at<float>(ws, lay.up), M, F, d, F, false, s);
    }
    launch_swiglu_f32(at<float>(ws, lay.gate), at<float>(ws, lay.up), at<float>(ws, lay.u), (long)M * F, s);
    ProfScope p(m, PK_DOWN, s);
    launch_gemm_f32(at<float>(ws, lay.u), Wf(m, base + 8), h, M, d, F, d, true, s);
  }
}

void run_layer(const dllm_model* m, int layer, int part, int B, int L, void* ws, const Layout& lay, hipStream_t s,
               const LayerRows* rows = nullptr) {
  if (m->cfg.dtype == DLLM_BF16)
    run_layer_bf16(m, layer, part, B, L, ws, lay, s, nullptr, nullptr, rows);
  else
    run_layer_f32(m, layer, part, B, L, ws, lay, s, rows);
}

// Buffers of the final norm and LM head: the residual h they read and their
// scratch (normed rows, the operand-order copy, the per-workgroup partials and
// ticket of the bf16 head; the logits of the float32 head).
struct HeadBufs {
  float* h;
  void* hb;
  bf16_t* hbf;
  float* logits;
  float* part_m;
  float* part_s;
  int32_t* part_i;
  int* ticket;
};

HeadBufs head_bufs(void* ws, const Layout& lay, const dllm_model_cfg& c) {
  HeadBufs b{};
  b.h = at<float>(ws, lay.h);
  b.hb = at<void>(ws, lay.hb);
  if (c.dtype == DLLM_F32) {
    b.logits = at<float>(ws, lay.logits);
  } else {
    b.hbf = at<bf16_t>(ws, lay.hbf);
    b.part_m = at<float>(ws, lay.part_m);
    b.part_s = at<float>(ws, lay.part_s);
    b.part_i = at<int32_t>(ws, lay.part_i);
    b.ticket = at<int>(ws, lay.ticket);
  }
  return b;
}

// Final norm and LM head on rows [row0, row0 + rows) of every sequence of
// hb.h ([B*L, d]); pend: split-K partials the last layer's down projection
// left pending (added to the head rows by the final norm; the other rows of h
// stay without them).
void run_head_bufs(const dllm_model* m, int B, int L, int row0, int rows, float* conf, int32_t* argmax,
                   float* logits, const HeadBufs& hb, hipStream_t s, const PendingResid* pend = nullptr) {
  const auto& c = m->cfg;
  const int nl = c.n_layers;
  const int R = B * rows;
  // bf16: up to HEAD_FRAG_ROWS head rows also go to an MFMA-operand-order copy
  // for the streaming head kernel
  bf16_t* hbf = c.dtype == DLLM_BF16 && R <= HEAD_FRAG_ROWS ? hb.hbf : nullptr;
  {
    ProfScope p(m, PK_NORM, s);
    // the head kernel's ticket is zeroed here (no memset node in a captured step)
    if (c.dtype == DLLM_BF16)
      launch_rmsnorm_head(hb.h, pend, static_cast<const bf16_t*>(W(m, 1 + 9 * nl)), static_cast<bf16_t*>(hb.hb), hbf,
                          B, rows, L, row0, c.d_model, c.rms_eps, hb.ticket, s);
    else
      launch_rmsnorm(hb.h, W(m, 1 + 9 * nl), hb.hb, c.dtype, B, rows, L, row0, c.d_model, c.rms_eps, s);
  }
  ProfScope p(m, PK_HEAD, s);
  if (c.dtype == DLLM_F32) {
    float* lg = logits ? logits : hb.logits;
    launch_gemm_f32(static_cast<const float*>(hb.hb), Wf(m, 2 + 9 * nl), lg, R, c.vocab, c.d_model, c.vocab, false,
                    s);
    launch_vocab_reduce_f32(lg, R, c.vocab, c.mask_id, conf, argmax, s);
  } else {
    HeadArgs a{};
    a.hb = static_cast<const bf16_t*>(hb.hb);
    a.hbf = hbf;
    a.W = m->head_tiled;
    a.R = R;
    a.V = c.vocab;
    a.d = c.d_model;
    a.mask_id = c.mask_id;
    a.conf = conf;
    a.argmax = argmax;
    a.logits = logits;
    a.part_m = hb.part_m;
    a.part_s = hb.part_s;
    a.part_i = hb.part_i;
    a.ticket = hb.ticket;
    launch_head_bf16(a, s);
  }
}

void run_head(const dllm_model* m, int B, int L, int row0, int rows, float* conf, int32_t* argmax, float* logits,
              void* ws, const Layout& lay, hipStream_t s, const PendingResid* pend = nullptr) {
  run_head_bufs(m, B, L, row0, rows, conf, argmax, logits, head_bufs(ws, lay, m->cfg), s, pend);
}

// ---------------------------------------------------------------- controller
void check_params(const dllm_cai_params* p) {
  require(p != nullptr, DLLM_EINVAL, "params is NULL");
  require((p->flags & ~(uint32_t)(DLLM_F_BLOCK_SCHED | DLLM_F_POS | DLLM_F_BUDGET | DLLM_F_GRIND | DLLM_F_FIXED)) == 0,
          DLLM_EINVAL, "unknown flag bits");
  require(p->block_len >= 1 && p->block_len <= 64, DLLM_EUNSUPPORTED, "block_len must be in [1, 64]");
  require(p->steps_per_block >= 0, DLLM_EINVAL, "steps_per_block must be >= 0");
  const double dv[] = {p->theta_s, p->theta_e, p->theta_e_step, p->theta_e_floor, p->warmup, p->clip_lo,
                       p->clip_hi, p->eta_bar, p->pos_factor[0], p->pos_factor[1], p->pos_factor[2],
                       p->pos_factor[3]};
  for (double v : dv) require(std::isfinite(v), DLLM_EINVAL, "non-finite controller constant");
  const float fv[] = {p->s_easy, p->s_hard, p->theta_fb};
  for (float v : fv) require(std::isfinite(v), DLLM_EINVAL, "non-finite controller constant");
  require(p->warmup >= 0.0 && p->warmup < 1.0, DLLM_EINVAL, "warmup must be in [0, 1)");
  require(p->clip_lo <= p->clip_hi, DLLM_EINVAL, "clip_lo > clip_hi");
  require(p->patience >= 1, DLLM_EINVAL, "patience must be >= 1");
  require(p->pos_edge[0] <= p->pos_edge[1] && p->pos_edge[1] <= p->pos_edge[2], DLLM_EINVAL,
          "pos_edge must be non-decreasing");
}

int steps_T(const dllm_cai_params* p) { return p->steps_per_block > 0 ? p->steps_per_block : p->block_len; }

// theta_b(t) in float64 (Boxes 3 and 4), b 1-based.
double block_threshold(const dllm_cai_params* p, int b, int t) {
  const int T = steps_T(p);
  const double wT = p->warmup * T;
  if ((double)t < wT) return p->theta_s;
  double te = p->theta_e;
  if (p->flags & DLLM_F_BLOCK_SCHED) te = std::max(p->theta_e - p->theta_e_step * (b - 1), p->theta_e_floor);
  const double u = ((double)t - wT) / ((double)T - wT);
  return te + 0.5 * (p->theta_s - te) * (1.0 + cos(M_PI * u));
}

void fill_commit_args(const dllm_cai_params* p, dllm_state* st, CommitArgs* a, int B, int P, int G, int block, int t,
                      int mask_id) {
  require(st && st->x && st->commit_step && st->reason && st->s && st->budget && st->ell && st->done, DLLM_EINVAL,
          "state has a NULL member");
  require(B >= 1 && B <= 16, DLLM_EUNSUPPORTED, "batch must be in [1, 16]");
  require(G >= 1 && G % p->block_len == 0, DLLM_ESHAPE, "G must be a positive multiple of block_len");
  require(P >= 0, DLLM_ESHAPE, "P must be >= 0");
  require(block >= 0 && block < G / p->block_len, DLLM_ESHAPE, "block index out of range");
  const int T = steps_T(p);
  require(t >= 0 && t < T, DLLM_ESHAPE, "step index out of range");
  a->x = st->x;
  a->commit_step = st->commit_step;
  a->reason = st->reason;
  a->sv = st->s;
  a->budget = st->budget;
  a->ell = st->ell;
  a->done = st->done;
  a->B = B;
  a->L = P + G;
  a->P = P;
  a->G = G;
  a->bl = p->block_len;
  a->g0 = block * p->block_len;
  a->t = t;
  a->T = T;
  a->mask_id = mask_id;
  const double tb = block_threshold(p, block + 1, t);
  for (int band = 0; band < 4; ++band) {
    double th = tb;
    if (p->flags & DLLM_F_POS) th = std::min(std::max(tb * p->pos_factor[band], p->clip_lo), p->clip_hi);
    a->thr[band] = (float)th;
  }
  for (int i = 0; i < 3; ++i) a->edge[i] = p->pos_edge[i];
  a->budget_on = (p->flags & DLLM_F_BUDGET) ? 1 : 0;
  a->grind_on = (p->flags & DLLM_F_GRIND) ? 1 : 0;
  a->s_easy = p->s_easy;
  a->s_hard = p->s_hard;
  a->p_easy = p->p_easy;
  a->p_hard = p->p_hard;
  a->b_easy = p->budget_easy;
  a->b_mid = p->budget_mid;
  a->b_hard = p->budget_hard;
  a->eta_bar = p->eta_bar;
  a->patience = p->patience;
  a->theta_fb = p->theta_fb;
  // fixed schedule: floor(bl / T) per step, one more in the first bl % T steps
  a->fixed = (p->flags & DLLM_F_FIXED) ? 1 : 0;
  a->fixed_k = a->fixed ? p->block_len / T + (t < p->block_len % T ? 1 : 0) : 0;
}

// Every layer on the B * Lq rows of h (see LayerRows; kv null: the full
// sequence with keys/values in the workspace).  Each layer's down-projection
// partials are added by the next layer's first norm; the last layer's are
// returned for the final norm, which adds them to the head rows only.
PendingResid run_layers(const dllm_model* m, int B, int L, int Lq, int pos0, void* kv, void* ws, const Layout& lay,
                        hipStream_t s) {
  const int nl = m->cfg.n_layers;
  PendingResid carry;
  for (int l = 0; l < nl; ++l) {
    LayerRows r{Lq, pos0, nullptr, nullptr};
    if (kv) r = cache_rows(m, kv, l, B, L, Lq, pos0);
    if (m->cfg.dtype == DLLM_BF16)
      run_layer_bf16(m, l, 2, B, L, ws, lay, s, &carry, &carry, &r);
    else
      run_layer_f32(m, l, 2, B, L, ws, lay, s, &r);
  }
  return carry;
}

// The full forward over all L positions, head on rows [row0, row0 + rows);
// with kv non-null every layer's keys/values are stored in the cache
// (a refresh step).
void forward_all(const dllm_model* m, const int32_t* x, int B, int L, int row0, int rows, float* conf,
                 int32_t* argmax, float* logits, void* ws, const Layout& lay, hipStream_t s, void* kv = nullptr,
                 bool rope = true) {
  {
    ProfScope p(m, PK_NORM, s);
    run_embed(m, x, B, L, 0, L, ws, lay, s, rope);
  }
  const PendingResid pend = run_layers(m, B, L, L, 0, kv, ws, lay, s);
  run_head(m, B, L, row0, rows, conf, argmax, logits, ws, lay, s, &pend);
}

// A cached step's forward: only rows [row0, row0 + rows) of each sequence go
// through the layers, attending over the cache (whose entries at those
// positions they overwrite); the head runs on all of them.
void forward_cached(const dllm_model* m, const int32_t* x, int B, int L, int row0, int rows, float* conf,
                    int32_t* argmax, float* logits, void* kv, void* ws, const Layout& lay, hipStream_t s,
                    bool rope = true) {
  {
    ProfScope p(m, PK_NORM, s);
    run_embed(m, x, B, L, row0, rows, ws, lay, s, rope);
  }
  const PendingResid pend = run_layers(m, B, L, rows, row0, kv, ws, lay, s);
  run_head(m, B, rows, 0, rows, conf, argmax, logits, ws, lay, s, &pend);
}

void check_cfg(const dllm_model_cfg* cfg) {
  require(cfg != nullptr, DLLM_EINVAL, "cfg is NULL");
  const auto& c = *cfg;
  require(c.n_layers >= 0 && c.d_model > 0 && c.n_heads > 0 && c.n_kv_heads > 0 && c.head_dim > 0 && c.d_ff > 0 &&
              c.vocab > 1,
          DLLM_EINVAL, "model dimensions must be positive");
  require(c.n_heads % c.n_kv_heads == 0, DLLM_EINVAL, "n_heads must be a multiple of n_kv_heads");
  require(c.mask_id >= 0 && c.mask_id < c.vocab, DLLM_EINVAL, "mask_id out of range");
  require(std::isfinite(c.rms_eps) && c.rms_eps > 0 && std::isfinite(c.rope_base) && c.rope_base > 0, DLLM_EINVAL,
          "rms_eps and rope_base must be positive");
  require(c.dtype == DLLM_F32 || c.dtype == DLLM_BF16, DLLM_EINVAL, "dtype must be DLLM_F32 or DLLM_BF16");
  if (c.dtype == DLLM_BF16)
    require(c.head_dim == 128 && c.d_model % 256 == 0 && c.d_ff % 128 == 0 && c.n_heads % 2 == 0 &&
                c.n_kv_heads % 2 == 0,
            DLLM_EUNSUPPORTED,
            "bf16 path needs head_dim 128, d_model % 256 == 0, d_ff % 128 == 0, even head counts");
  else
    require((c.head_dim == 64 || c.head_dim == 128), DLLM_EUNSUPPORTED, "fp32 path needs head_dim 64 or 128");
  if (c.dtype == DLLM_BF16)
    require(head_bf16_packed_bytes(c.vocab, c.d_model) <= 0x7fffffffu, DLLM_EUNSUPPORTED,
            "bf16 LM head larger than 2 GiB");
}

// Bytes of the packed layer-weight copies, and (off non-null) each copy's
// element offset: [layer * 4 + {0: q/k/v, 1: output, 2: gate/up, 3: down}].
size_t packed_layout(const dllm_model* m, std::vector<size_t>* off) {
  const int nl = m->cfg.n_layers;
  if (off) off->assign((size_t)nl * 4, 0);
  size_t total = 0;
  for (int l = 0; l < nl; ++l)
    for (int w = 0; w < 4; ++w) {
      const GemmArgs g = layer_gemm(m, l, w);
      if (off) (*off)[(size_t)l * 4 + w] = total / sizeof(bf16_t);
      total += align256(gemm_packed_bytes(g.N, g.K));
    }
  return std::max<size_t>(total, 256);
}

// The step's error word, as the commit kernel reports it (bits above bit 0 of
// the block-finished word).
void raise_step_errors(int flag) {
  const int e = flag >> 1;
  if (e & ERR_TOKEN_RANGE) fail(DLLM_EINVAL, "a token id is outside [0, vocab)");
  if (e & ERR_V_RANGE)
    fail(DLLM_EUNSUPPORTED, "a value of v is beyond IEEE half's range (stored as +-65504 for the attention)");
}

int finish(const ApiError& e) {
  g_last_error = e.msg;
  return e.code;
}

}  // namespace

// ---------------------------------------------------------------- static scratch
// Scratch of dllm_head_noalloc: one array per GPU, resident until the process
// ends.  Host code never uses the name (a host-side stand-in); the device
// address comes from hipGetSymbolAddress, taken once per device.
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

// The current device's copy of `scratch` (looked up on its first use on that
// device, with the device current).
void* device_scratch() {
  int dev = -1;
  hip_check(hipGetDevice(&dev), "hipGetDevice");
  require(dev >= 0 && dev < MAX_DEVICES, DLLM_EUNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    require(p != nullptr, DLLM_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

// The head's scratch carved out of `base` (nullptr: sizes only); returns the bytes.
size_t noalloc_head_layout(const dllm_model_cfg& c, int R, char* base, HeadBufs* b) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* at = base ? base + off : nullptr;
    off += align256(bytes);
    return at;
  };
  const size_t act = c.dtype == DLLM_F32 ? 4 : 2;
  b->hb = take((size_t)R * c.d_model * act);
  if (c.dtype == DLLM_F32) {
    b->logits = reinterpret_cast<float*>(take((size_t)R * c.vocab * 4));
  } else {
    const size_t slots = (size_t)head_bf16_tiles(c.vocab) * R * 4;
    b->hbf = reinterpret_cast<bf16_t*>(take((size_t)HEAD_FRAG_ROWS * c.d_model * 2));
    b->part_m = reinterpret_cast<float*>(take(slots));
    b->part_s = reinterpret_cast<float*>(take(slots));
    b->part_i = reinterpret_cast<int32_t*>(take(slots));
    b->ticket = reinterpret_cast<int*>(take(4));
  }
  return off;
}
}  // namespace

#define API_BEGIN \
  g_last_error.clear(); \
  try {
#define API_END                                   \
  }                                               \
  catch (const ApiError& e) {                     \
    return finish(e);                             \
  }                                               \
  catch (const HipError& e) {                     \
    g_last_error = e.what();                      \
    return DLLM_EHIP;                             \
  }                                               \
  catch (const std::exception& e) {               \
    g_last_error = e.what();                      \
    return DLLM_EINVAL;                           \
  }                                               \
  return DLLM_OK;

extern "C" {

const char* dllm_last_error(void) { return g_last_error.c_str(); }

int dllm_model_buffer_size(const dllm_model_cfg* cfg, size_t* bytes) {
  API_BEGIN
  require(bytes != nullptr, DLLM_EINVAL, "bytes is NULL");
  check_cfg(cfg);
  *bytes = cfg->dtype == DLLM_BF16 ? align256(head_bf16_packed_bytes(cfg->vocab, cfg->d_model)) : 0;
  API_END
}

int dllm_model_create(const dllm_model_cfg* cfg, const void* const* weights, int32_t n_weights, void* model_buf,
                      size_t model_buf_bytes, void* stream, dllm_model** out) {
  API_BEGIN
  require(weights && out, DLLM_EINVAL, "NULL argument");
  check_cfg(cfg);
  const auto& c = *cfg;
  require(n_weights == 3 + 9 * c.n_layers, DLLM_EINVAL, "n_weights must be 3 + 9 * n_layers");
  for (int i = 0; i < n_weights; ++i) require(weights[i] != nullptr, DLLM_EINVAL, "NULL weight pointer");
  if (c.dtype == DLLM_BF16) {
    const size_t need = align256(head_bf16_packed_bytes(c.vocab, c.d_model));
    require(model_buf != nullptr, DLLM_EINVAL, "model_buf is NULL (a bf16 model keeps its LM-head copy there)");
    require(((uintptr_t)model_buf & 255) == 0, DLLM_EINVAL, "model_buf must be 256-byte aligned");
    require(model_buf_bytes >= need, DLLM_ENOMEM, "model_buf too small: need " + std::to_string(need) + " bytes");
  }
  auto* m = new dllm_model();
  m->cfg = c;
  m->w.assign(weights, weights + n_weights);
  try {
    hip_check(hipHostMalloc((void**)&m->step_flag, sizeof(int32_t), hipHostMallocMapped | hipHostMallocCoherent),
              "hipHostMalloc");
    *m->step_flag = 0;
    hip_check(hipHostGetDevicePointer((void**)&m->step_flag_dev, m->step_flag, 0), "hipHostGetDevicePointer");
    if (c.dtype == DLLM_BF16) {
      // stream-ordered after the caller's writes of lm_head on that stream
      m->head_tiled = static_cast<bf16_t*>(model_buf);
      launch_pack_head_bf16(static_cast<const bf16_t*>(m->w[2 + 9 * c.n_layers]), m->head_tiled, c.vocab, c.d_model,
                            (hipStream_t)stream);
    }
  } catch (...) {
    if (m->step_flag) (void)hipHostFree(m->step_flag);
    delete m;
    throw;
  }
  *out = m;
  API_END
}

int dllm_model_destroy(dllm_model* m) {
  API_BEGIN
  if (!m) return DLLM_OK;
  for (auto& e : m->events) {
    (void)hipEventDestroy(e.start);
    (void)hipEventDestroy(e.stop);
  }
  if (m->step_flag) (void)hipHostFree(m->step_flag);
  delete m;
  API_END
}

int dllm_model_packed_size(const dllm_model* m, size_t* bytes) {
  API_BEGIN
  check_model(m);
  require(bytes != nullptr, DLLM_EINVAL, "bytes is NULL");
  require(m->cfg.dtype == DLLM_BF16, DLLM_EUNSUPPORTED, "packed weights are for bf16 models");
  *bytes = packed_layout(m, nullptr);
  API_END
}

int dllm_model_pack_weights(dllm_model* m, void* buf, size_t bytes, void* stream) {
  API_BEGIN
  check_model(m);
  require(m->cfg.dtype == DLLM_BF16, DLLM_EUNSUPPORTED, "packed weights are for bf16 models");
  std::vector<size_t> off;
  const size_t need = packed_layout(m, &off);
  require(buf != nullptr, DLLM_EINVAL, "buf is NULL");
  require(((uintptr_t)buf & 255) == 0, DLLM_EINVAL, "buf must be 256-byte aligned");
  require(bytes >= need, DLLM_ENOMEM, "packed-weight buffer too small: need " + std::to_string(need) + " bytes");
  bf16_t* dst = static_cast<bf16_t*>(buf);
  const int nl = m->cfg.n_layers;
  // stream-ordered after the caller's writes of the weights on that stream
  for (int l = 0; l < nl; ++l)
    for (int w = 0; w < 4; ++w)
      launch_pack_gemm_weights(layer_gemm(m, l, w), dst + off[(size_t)l * 4 + w], (hipStream_t)stream);
  m->packed_off = off;
  m->packed = dst;
  API_END
}

int dllm_workspace_size(const dllm_model* m, int32_t B, int32_t L, int32_t rows, size_t* bytes) {
  API_BEGIN
  check_model(m);
  require(bytes != nullptr, DLLM_EINVAL, "bytes is NULL");
  require(B >= 1 && L >= 1 && rows >= 0 && rows <= L, DLLM_ESHAPE, "bad sizes");
  *bytes = make_layout(m->cfg, B, L, rows).total;
  API_END
}

int dllm_workspace_layout(const dllm_model* m, int32_t B, int32_t L, int32_t rows, dllm_ws_layout* out) {
  API_BEGIN
  check_model(m);
  require(out != nullptr, DLLM_EINVAL, "out is NULL");
  require(B >= 1 && L >= 1 && rows >= 0 && rows <= L, DLLM_ESHAPE, "bad sizes");
  const Layout l = make_layout(m->cfg, B, L, rows);
  out->total = l.total;
  out->h = l.h;
  out->a_attn = l.a_attn;
  out->q = l.q;
  out->k = l.k;
  out->vt = l.vt;
  out->attn = l.attn;
  out->a_mlp = l.a_mlp;
  out->u = l.u;
  out->hb = l.hb;
  API_END
}

int dllm_embed(const dllm_model* m, const int32_t* x, int32_t B, int32_t L, void* ws, size_t ws_bytes,
               void* stream) {
  API_BEGIN
  check_model(m);
  require(x != nullptr, DLLM_EINVAL, "x is NULL");
  Layout lay;
  check_ws(m, B, L, 0, ws, ws_bytes, &lay);
  run_embed(m, x, B, L, 0, L, ws, lay, (hipStream_t)stream);
  API_END
}

int dllm_embed_rows(const dllm_model* m, const int32_t* x, int32_t B, int32_t L, int32_t row0, int32_t rows,
                    void* ws, size_t ws_bytes, void* stream) {
  API_BEGIN
  check_model(m);
  require(x != nullptr, DLLM_EINVAL, "x is NULL");
  require(row0 >= 0 && rows >= 1 && row0 + rows <= L, DLLM_ESHAPE, "rows out of range");
  Layout lay;
  check_ws(m, B, L, rows, ws, ws_bytes, &lay);
  run_embed(m, x, B, L, row0, rows, ws, lay, (hipStream_t)stream);
  API_END
}

int dllm_kv_cache_size(const dllm_model* m, int32_t B, int32_t L, size_t* bytes) {
  API_BEGIN
  check_model(m);
  require(bytes != nullptr, DLLM_EINVAL, "bytes is NULL");
  require(B >= 1 && L >= 1, DLLM_ESHAPE, "bad sizes");
  *bytes = kv_cache_bytes(m->cfg, B, L);
  API_END
}

int dllm_layer_kv(const dllm_model* m, int32_t layer, int32_t part, int32_t B, int32_t L, int32_t row0,
                  int32_t rows, void* kv, size_t kv_bytes, void* ws, size_t ws_bytes, void* stream) {
  API_BEGIN
  check_model(m);
  require(layer >= 0 && layer < m->cfg.n_layers, DLLM_EINVAL, "layer out of range");
  require(part >= 0 && part <= 2, DLLM_EINVAL, "part must be 0, 1 or 2");
  require(row0 >= 0 && rows >= 1 && row0 + rows <= L, DLLM_ESHAPE, "rows out of range");
  check_kv(m, B, L, kv, kv_bytes);
  Layout lay;
  check_ws(m, B, L, rows == L ? 0 : rows, ws, ws_bytes, &lay);
  const LayerRows r = cache_rows(m, kv, layer, B, L, rows, row0);
  run_layer(m, layer, part, B, L, ws, lay, (hipStream_t)stream, &r);
  API_END
}

int dllm_layer(const dllm_model* m, int32_t layer, int32_t part, int32_t B, int32_t L, void* ws, size_t ws_bytes,
               void* stream) {
  API_BEGIN
  check_model(m);
  require(layer >= 0 && layer < m->cfg.n_layers, DLLM_EINVAL, "layer out of range");
  require(part >= 0 && part <= 2, DLLM_EINVAL, "part must be 0, 1 or 2");
  Layout lay;
  check_ws(m, B, L, 0, ws, ws_bytes, &lay);
  run_layer(m, layer, part, B, L, ws, lay, (hipStream_t)stream);
  API_END
}

int dllm_head(const dllm_model* m, int32_t B, int32_t L, int32_t row0, int32_t rows, float* conf, int32_t* argmax,
              float* logits, void* ws, size_t ws_bytes, void* stream) {
  API_BEGIN
  check_model(m);
  require(conf && argmax, DLLM_EINVAL, "conf/argmax is NULL");
  require(row0 >= 0 && rows >= 1 && row0 + rows <= L, DLLM_ESHAPE, "rows out of range");
  Layout lay;
  check_ws(m, B, L, rows, ws, ws_bytes, &lay);
  run_head(m, B, L, row0, rows, conf, argmax, logits, ws, lay, (hipStream_t)stream);
  API_END
}

int dllm_head_noalloc(const dllm_model* m, const float* h, int32_t B, int32_t L, int32_t row0, int32_t rows,
                      float* conf, int32_t* argmax, float* logits, void* stream) {
  API_BEGIN
  check_model(m);
  require(h && conf && argmax, DLLM_EINVAL, "h/conf/argmax is NULL");
  require(((uintptr_t)h & 15) == 0, DLLM_EINVAL, "h must be 16-byte aligned");
  require(B >= 1 && B <= 16, DLLM_EUNSUPPORTED, "batch must be in [1, 16]");
  require(L >= 1 && row0 >= 0 && rows >= 1 && row0 + rows <= L, DLLM_ESHAPE, "rows out of range");
  if (m->cfg.dtype == DLLM_BF16)
    require((long)B * rows <= head_bf16_max_rows(), DLLM_EUNSUPPORTED, "B * rows exceeds the LM-head kernel limit");
  HeadBufs hb{};
  const size_t need = noalloc_head_layout(m->cfg, B * rows, nullptr, &hb);
  require(need <= NOALLOC_SCRATCH_BYTES, DLLM_ENOMEM,
          "dllm_head_noalloc needs " + std::to_string(need) + " bytes of scratch; the static scratch holds " +
              std::to_string(NOALLOC_SCRATCH_BYTES));
  noalloc_head_layout(m->cfg, B * rows, static_cast<char*>(device_scratch()), &hb);
  hb.h = const_cast<float*>(h);  // read only: no split-K partials are pending here
  run_head_bufs(m, B, L, row0, rows, conf, argmax, logits, hb, (hipStream_t)stream);
  API_END
}

int dllm_forward(const dllm_model* m, const int32_t* x, int32_t B, int32_t L, int32_t row0, int32_t rows,
                 float* conf, int32_t* argmax, float* logits, void* ws, size_t ws_bytes, void* stream) {
  API_BEGIN
  check_model(m);
  require(x && conf && argmax, DLLM_EINVAL, "NULL argument");
  require(row0 >= 0 && rows >= 1 && row0 + rows <= L, DLLM_ESHAPE, "rows out of range");
  Layout lay;
  check_ws(m, B, L, rows, ws, ws_bytes, &lay);
  forward_all(m, x, B, L, row0, rows, conf, argmax, logits, ws, lay, (hipStream_t)stream);
  API_END
}

int dllm_forward_kv(const dllm_model* m, const int32_t* x, int32_t B, int32_t L, int32_t row0, int32_t rows,
                    int32_t refresh, float* conf, int32_t* argmax, float* logits, void* kv, size_t kv_bytes, void* ws,
                    size_t ws_bytes, void* stream) {
  API_BEGIN
  check_model(m);
  require(x && conf && argmax, DLLM_EINVAL, "NULL argument");
  require(row0 >= 0 && rows >= 1 && row0 + rows <= L, DLLM_ESHAPE, "rows out of range");
  check_kv(m, B, L, kv, kv_bytes);
  Layout lay;
  check_ws(m, B, L, rows, ws, ws_bytes, &lay);
  if (refresh)
    forward_all(m, x, B, L, row0, rows, conf, argmax, logits, ws, lay, (hipStream_t)stream, kv);
  else
    forward_cached(m, x, B, L, row0, rows, conf, argmax, logits, kv, ws, lay, (hipStream_t)stream);
  API_END
}

int dllm_state_init(int32_t mask_id, const int32_t* prompt, int32_t B, int32_t P, int32_t G, dllm_state* st,
                    void* stream) {
  API_BEGIN
  require(mask_id >= 0, DLLM_EINVAL, "mask_id must be >= 0");
  require(st && st->x && st->commit_step && st->reason && st->s && st->budget && st->ell && st->done, DLLM_EINVAL,
          "state has a NULL member");
  require(B >= 1 && B <= 16 && P >= 0 && G >= 1, DLLM_ESHAPE, "bad sizes");
  require(P == 0 || prompt != nullptr, DLLM_EINVAL, "prompt is NULL");
  launch_state_init(prompt, st->x, st->commit_step, st->reason, st->s, st->budget, st->ell, st->done, B, P, G,
                    mask_id, nullptr, (hipStream_t)stream);
  API_END
}

int dllm_commit(const dllm_cai_params* p, dllm_state* st, const float* conf, const int32_t* argmax, int32_t B,
                int32_t P, int32_t G, int32_t block, int32_t t, int32_t mask_id, int32_t* all_done, void* stream) {
  API_BEGIN
  check_params(p);
  require(conf && argmax, DLLM_EINVAL, "conf/argmax is NULL");
  CommitArgs a{};
  fill_commit_args(p, st, &a, B, P, G, block, t, mask_id);
  a.conf = conf;
  a.argmax = argmax;
  a.all_done = all_done;
  launch_commit(a, (hipStream_t)stream);
  API_END
}

namespace {
// One denoising step.  kv null: the full forward; else a refresh step (the
// full forward storing the cache) when refresh is set, a cached step otherwise.
// One denoising step; with seq > 0 the commit also publishes its done/error
// word to the model's pinned step flag under that sequence number (wait_step).
void step_impl(const dllm_model* m, const dllm_cai_params* p, dllm_state* st, int B, int P, int G, int block, int t,
               float* conf_out, int32_t* argmax_out, void* ws, const Layout& lay, hipStream_t s, void* kv = nullptr,
               bool refresh = true, bool rope = true, int seq = 0) {
  CommitArgs a{};
  fill_commit_args(p, st, &a, B, P, G, block, t, m->cfg.mask_id);
  const int bl = p->block_len;
  float* conf = conf_out ? conf_out : at<float>(ws, lay.conf);
  int32_t* arg = argmax_out ? argmax_out : at<int32_t>(ws, lay.argmax);
  if (kv && !refresh)
    forward_cached(m, st->x, B, P + G, P + block * bl, bl, conf, arg, nullptr, kv, ws, lay, s, rope);
  else
    forward_all(m, st->x, B, P + G, P + block * bl, bl, conf, arg, nullptr, ws, lay, s, kv, rope);
  a.conf = conf;
  a.argmax = arg;
  a.all_done = at<int32_t>(ws, lay.all_done);
  a.err = at<int>(ws, lay.err);
  if (seq > 0) {
    a.host_flag = m->step_flag_dev;
    a.seq = seq;
  }
  ProfScope pr(m, PK_COMMIT, s);
  launch_commit(a, s);
}

// Sequence number for the next published step (1 .. 2^23 - 1, wrapping).
int next_seq(const dllm_model* m) {
  auto* mm = const_cast<dllm_model*>(m);
  mm->step_seq = mm->step_seq % 0x7fffff + 1;
  return mm->step_seq;
}

// The done/error word of the step published under seq: the host polls the
// pinned flag the commit kernel stores to (it sees the word microseconds after
// the store; a stream synchronisation after a device-to-host copy costs the
// GPU a few hundred microseconds of idle time per step).  A word that has not
// arrived after 20 ms falls back to synchronising the stream, which returns
// once the step has run or reports its error.
int wait_step(const dllm_model* m, hipStream_t s, int seq) {
  volatile int32_t* f = m->step_flag;
  const auto t0 = std::chrono::steady_clock::now();
  for (long i = 1;; ++i) {
    const int v = *f;
    if ((v >> 8) == seq) return v & 0xff;
    if ((i & 1023) == 0 && std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(20)) break;
    __builtin_ia32_pause();
  }
  hip_check(hipStreamSynchronize(s), "hipStreamSynchronize");
  const int v = *f;
  if ((v >> 8) != seq) fail(DLLM_EHIP, "the step's done flag was not published");
  return v & 0xff;
}
}  // namespace

int dllm_step(const dllm_model* m, const dllm_cai_params* p, dllm_state* st, int32_t B, int32_t P, int32_t G,
              int32_t block, int32_t t, float* conf_out, int32_t* argmax_out, int32_t* all_done_host, void* ws,
              size_t ws_bytes, void* stream) {
  API_BEGIN
  check_model(m);
  check_params(p);
  Layout lay;
  check_ws(m, B, P + G, p->block_len, ws, ws_bytes, &lay);
  hipStream_t s = (hipStream_t)stream;
  const int seq = all_done_host ? next_seq(m) : 0;
  step_impl(m, p, st, B, P, G, block, t, conf_out, argmax_out, ws, lay, s, nullptr, true, true, seq);
  if (all_done_host) {
    const int flag = wait_step(m, s, seq);
    *all_done_host = flag & 1;
    raise_step_errors(flag);
  }
  API_END
}

int dllm_step_kv(const dllm_model* m, const dllm_cai_params* p, int32_t refresh, dllm_state* st, int32_t B,
                 int32_t P, int32_t G, int32_t block, int32_t t, float* conf_out, int32_t* argmax_out,
                 int32_t* all_done_host, void* kv, size_t kv_bytes, void* ws, size_t ws_bytes, void* stream) {
  API_BEGIN
  check_model(m);
  check_params(p);
  check_kv(m, B, P + G, kv, kv_bytes);
  Layout lay;
  check_ws(m, B, P + G, p->block_len, ws, ws_bytes, &lay);
  hipStream_t s = (hipStream_t)stream;
  const int seq = all_done_host ? next_seq(m) : 0;
  step_impl(m, p, st, B, P, G, block, t, conf_out, argmax_out, ws, lay, s, kv, refresh != 0, true, seq);
  if (all_done_host) {
    const int flag = wait_step(m, s, seq);
    *all_done_host = flag & 1;
    raise_step_errors(flag);
  }
  API_END
}

namespace {
// The block loop of dllm_generate / dllm_generate_kv (refresh_every 0: no cache).
void generate_impl(const dllm_model* m, const dllm_cai_params* p, const int32_t* prompt, int B, int P, int G,
                   dllm_state* st, int32_t* forwards_host, int32_t* total_forwards, float* conf_trace,
                   int32_t* argmax_trace, void* kv, int refresh_every, void* ws, const Layout& lay, hipStream_t s) {
  const int bl = p->block_len, nb = G / bl, T = steps_T(p);
  launch_state_init(prompt, st->x, st->commit_step, st->reason, st->s, st->budget, st->ell, st->done, B, P, G,
                    m->cfg.mask_id, at<int>(ws, lay.err), s);
  {  // positions are fixed for the whole decode: one RoPE table
    ProfScope pr(m, PK_NORM, s);
    launch_rope_table(at<float>(ws, lay.cosb), at<float>(ws, lay.sinb), P + G, m->cfg.head_dim, m->cfg.rope_base,
                      nullptr, s);
  }
  int total = 0;
  for (int blk = 0; blk < nb; ++blk) {
    int n = 0;
    for (int t = 0; t < T; ++t) {
      float* ct = conf_trace ? conf_trace + ((size_t)blk * T + t) * B * bl : nullptr;
      int32_t* at_ = argmax_trace ? argmax_trace + ((size_t)blk * T + t) * B * bl : nullptr;
      const int seq = next_seq(m);
      step_impl(m, p, st, B, P, G, blk, t, ct, at_, ws, lay, s, kv, refresh_every == 0 || t % refresh_every == 0,
                false, seq);
      ++n;
      const int flag = wait_step(m, s, seq);
      raise_step_errors(flag);
      if (flag & 1) break;
    }
    if (forwards_host) forwards_host[blk] = n;
    total += n;
  }
  hip_check(hipStreamSynchronize(s), "hipStreamSynchronize");  // the last commit has returned
  if (total_forwards) *total_forwards = total;
}
}  // namespace

int dllm_generate(const dllm_model* m, const dllm_cai_params* p, const int32_t* prompt, int32_t B, int32_t P,
                  int32_t G, dllm_state* st, int32_t* forwards_host, int32_t* total_forwards, float* conf_trace,
                  int32_t* argmax_trace, void* ws, size_t ws_bytes, void* stream) {
  API_BEGIN
  check_model(m);
  check_params(p);
  require(G >= 1 && G % p->block_len == 0, DLLM_ESHAPE, "G must be a positive multiple of block_len");
  require(P >= 0 && (P == 0 || prompt), DLLM_EINVAL, "bad prompt");
  Layout lay;
  check_ws(m, B, P + G, p->block_len, ws, ws_bytes, &lay);
  generate_impl(m, p, prompt, B, P, G, st, forwards_host, total_forwards, conf_trace, argmax_trace, nullptr, 0, ws,
                lay, (hipStream_t)stream);
  API_END
}

int dllm_generate_kv(const dllm_model* m, const dllm_cai_params* p, int32_t refresh_every, const int32_t* prompt,
                     int32_t B, int32_t P, int32_t G, dllm_state* st, int32_t* forwards_host, int32_t* total_forwards,
                     float* conf_trace, int32_t* argmax_trace, void* kv, size_t kv_bytes, void* ws, size_t ws_bytes,
                     void* stream) {
  API_BEGIN
  check_model(m);
  check_params(p);
  require(refresh_every >= 1, DLLM_EINVAL, "refresh_every must be >= 1");
  require(G >= 1 && G % p->block_len == 0, DLLM_ESHAPE, "G must be a positive multiple of block_len");
  require(P >= 0 && (P == 0 || prompt), DLLM_EINVAL, "bad prompt");
  check_kv(m, B, P + G, kv, kv_bytes);
  Layout lay;
  check_ws(m, B, P + G, p->block_len, ws, ws_bytes, &lay);
  generate_impl(m, p, prompt, B, P, G, st, forwards_host, total_forwards, conf_trace, argmax_trace, kv, refresh_every,
                ws, lay, (hipStream_t)stream);
  API_END
}

int dllm_prof_enable(dllm_model* m, int32_t enable) {
  API_BEGIN
  check_model(m);
  require(enable >= 0 && enable < 256, DLLM_EINVAL, "enable must be a bit mask of kinds 0..7");
  m->prof_mask = (uint32_t)enable;
  m->n_events = 0;
  for (auto& c : m->prof_seen) c = 0;
  API_END
}

int dllm_prof_every(dllm_model* m, int32_t every) {
  API_BEGIN
  check_model(m);
  require(every >= 1, DLLM_EINVAL, "every must be >= 1");
  m->prof_every = every;
  for (auto& c : m->prof_seen) c = 0;
  API_END
}

int dllm_prof_read(dllm_model* m, int32_t kind, double* total_ms, int64_t* launches) {
  API_BEGIN
  check_model(m);
  require(total_ms && launches, DLLM_EINVAL, "NULL argument");
  double tot = 0;
  int64_t n = 0;
  for (size_t i = 0; i < m->n_events; ++i) {
    const ProfEvent& e = m->events[i];
    if (e.kind != kind) continue;
    hip_check(hipEventSynchronize(e.stop), "hipEventSynchronize");
    float ms = 0;
    hip_check(hipEventElapsedTime(&ms, e.start, e.stop), "hipEventElapsedTime");
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  API_END
}

}  // extern "C"
