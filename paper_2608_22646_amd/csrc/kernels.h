// Internal launchers of the dllm HIP kernels (not part of the C ABI).
#pragma once
#include "common.h"

namespace dllm {

// ---- k_misc.hip ------------------------------------------------------------
// Bits of the workspace's error word, set by kernels that meet an input they
// cannot represent and reported (then cleared) by the commit kernel.
enum { ERR_TOKEN_RANGE = 1, ERR_V_RANGE = 2 };
// h[b*rows + i, :] = float(E[x[b*L + row0 + i], :]) for b < B, i < rows.  An id
// outside [0, V) gathers a zero row and sets ERR_TOKEN_RANGE in *err.  The
// nzero ints at zero (the forward's attention tickets) are set to 0.
void launch_embed(const int32_t* x, const void* E, int dtype, float* h, int B, int rows, int L, int row0, int d,
                  int V, int* err, hipStream_t s, int* zero = nullptr, int nzero = 0);
// cos/sin [L, hd/2] of pos * base^(-2j/hd), evaluated in float64, stored float32;
// a non-null err word is cleared first (a forward starts with a clean word).
void launch_rope_table(float* cosb, float* sinb, int L, int hd, double base, int* err, hipStream_t s);
// out[b*rows + i, :] = act(RMSNorm(h[b*L + row0 + i, :]) * g) for b < B, i < rows.
void launch_rmsnorm(const float* h, const void* g, void* out, int dtype, int B, int rows, int L, int row0,
                    int d, float eps, hipStream_t s);
// Decoding state initialisation (see dllm_state_init); a non-null err word is
// cleared as well.
void launch_state_init(const int32_t* prompt, int32_t* x, int32_t* commit_step, int8_t* reason, float* sv,
                       int32_t* budget, int32_t* ell, int32_t* done, int B, int P, int G, int mask_id,
                       int* err, hipStream_t s);

// ---- fp32 path (k_f32.hip) -------------------------------------------------
// C[M, N] (+)= A[M, K] W[N, K]^T, all float32 row-major, C row stride ldc.
void launch_gemm_f32(const float* A, const float* W, float* C, int M, int N, int K, int ldc, bool accumulate,
                     hipStream_t s);
// Split raw projections [B*Lq, (Hq + 2 Hkv) hd] of the rows at positions pos0 ..
// pos0 + Lq - 1 of each sequence into q [B, Hq, Lq, hd] and k [B, Hkv, L, hd]
// (RoPE applied) and v^T [B, Hkv, hd, L] (k, v^T at those positions).
void launch_rope_split_f32(const float* raw, const float* cosb, const float* sinb, float* q, float* k,
                           float* vt, int B, int Lq, int L, int pos0, int Hq, int Hkv, int hd, hipStream_t s);
// out[i] = silu(gate[i]) * up[i]
void launch_swiglu_f32(const float* gate, const float* up, float* out, long n, hipStream_t s);
// Non-causal attention, float32, of Lq queries per sequence (q [B, Hq, Lq, hd])
// over L keys (k [B, Hkv, L, hd], v^T [B, Hkv, hd, L]): out[b*Lq + l, h*hd + j].
void launch_attn_f32(const float* q, const float* k, const float* vt, float* out, int B, int Lq, int L, int Hq,
                     int Hkv, int hd, hipStream_t s);
// Per row of logits [R, V]: conf = 1 / sum exp(l - max), argmax (lowest index), mask_id excluded.
void launch_vocab_reduce_f32(const float* logits, int R, int V, int mask_id, float* conf, int32_t* argmax,
                             hipStream_t s);

// ---- bf16 path -------------------------------------------------------------
enum GemmEpi { EPI_QKV_ROPE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_STORE = 3 };

struct GemmArgs {
  int epi;
  int M, N, K;              // N counts output columns of the virtual B (gate and up both counted)
  const bf16_t* A;          // [M, K]
  const bf16_t* W0;         // q / gate / plain weight [*, K]
  const bf16_t* W1;         // k / up
  const bf16_t* W2;         // v
  int n0, n1;               // rows of W0 and W1 (QKV: Hq*hd, Hkv*hd)
  // epilogue targets
  float* resid;             // EPI_RESID: [M, N] float32, += result
  bf16_t* out;              // EPI_SWIGLU: [M, N/2]; EPI_STORE: [M, N]
  bf16_t* q; bf16_t* k; f16_t* vt;   // EPI_QKV_ROPE (v^T holds the bf16 values as IEEE half)
  const float* cosb; const float* sinb;
  // EPI_QKV_ROPE: row m = b Lq + i holds position pos0 + i of sequence b; q is
  // [B, Hq, Lq, hd], k [B, Hkv, L, hd] and v^T [B, Hkv, hd, L] are written at
  // that position (a full forward: Lq = L, pos0 = 0)
  int B, L, Hq, Hkv, Lq, pos0;
  // split-K scratch (float32 partials [split, M, N]) from the workspace
  float* splitk_buf;
  // optional packed copy of Bv (launch_pack_gemm_weights): launches of at most
  // 128 rows then stream it instead of the row-major tensors
  const bf16_t* Wp;
  // EPI_QKV_ROPE: error word; a v value beyond IEEE half's range is stored as
  // +-65504 and sets ERR_V_RANGE
  int* err;
};
int device_cu_count();  // compute units of the current device (256 if it cannot be queried)
// Split-K partial tiles of a residual GEMM whose reduction into the residual
// has been left to the next RMSNorm (split 0: nothing pending).
struct PendingResid {
  const float* part = nullptr;  // [split, M, N] float32
  int split = 0;
};
// With defer non-null, a split-K residual GEMM of more than 128 rows leaves its
// partials pending there instead of launching the reduction (defer->split = 0
// otherwise).
void launch_gemm_bf16(const GemmArgs& a, hipStream_t s, PendingResid* defer = nullptr);
// Completes a deferred residual update and normalises in one pass, for every
// row m < M (bf16 model, d % 4 == 0, d <= 8192):
//   h[m, :] += sum_z part[z, m, :]   (z in order, as the split-K reduction does)
//   out[m, :] = bf16(RMSNorm(h[m, :]) * g)
// Rows up to which the split-K partials of the register-direct GEMM (1 .. 16
// of them) are left pending for the next norm, and the fused kernel runs one
// 1024-thread workgroup per row (d <= 8192).
constexpr int RESID_NORM_WIDE_ROWS = 64;
void launch_resid_rmsnorm(float* h, const PendingResid& pend, const bf16_t* g, bf16_t* out, int M, int d, float eps,
                          hipStream_t s);
// Packed copy of a GEMM's virtual weight matrix (g's W0/W1/W2, n0, n1, N, K,
// epi) in the LM head's tiled operand order, rows padded to 256.
size_t gemm_packed_bytes(int N, int K);
void launch_pack_gemm_weights(const GemmArgs& g, bf16_t* out, hipStream_t s);
// Bytes of split-K scratch a launch of this shape needs (0 if it does not split).
size_t gemm_bf16_splitk_bytes(int M, int N, int K, int epi);

// Non-causal attention of Lq queries per sequence (q [B, Hq, Lq, 128]) over L
// keys (k [B, Hkv, L, 128], v^T [B, Hkv, 128, L] as IEEE half):
// out[b*Lq + l, h*128 + j] (bf16).  With split_part (attn_split_bytes(B, Hq)
// bytes) and split_ticket (B * Hq ints, zero; left zero) a launch of at most 32
// queries per sequence splits the keys of each head over several workgroups.
size_t attn_split_bytes(int B, int Hq);
void launch_attn_bf16(const bf16_t* q, const bf16_t* k, const f16_t* vt, bf16_t* out, int B, int Lq, int L, int Hq,
                      int Hkv, hipStream_t s, float* split_part = nullptr, int* split_ticket = nullptr);

// The bf16 LM head is read from a tiled copy: vocabulary tiles of HEAD_TILE rows,
// each stored as d/64 consecutive [HEAD_TILE, 64] blocks, rows past V zero;
// inside a block, each 32-row x 16-k MFMA A operand is 1 KiB in lane order.
constexpr int HEAD_TILE = 256;
// Head-row counts up to HEAD_FRAG_ROWS use the streaming LM-head kernel, which
// reads the normed rows from a copy in MFMA B-operand order: for 16-k slice s,
// lane l = row + 32 * ((k / 8) % 2) holds bf16 k = 16 s + 8 (l / 32) .. +7
// (rows >= R unused), 1 KiB per slice.
constexpr int HEAD_FRAG_ROWS = 32;
// Final RMSNorm of the head rows (bf16 model, d % 4 == 0, d <= 8192): out[B*rows,
// d] row-major as launch_rmsnorm, and, when outf is non-null (B * rows <=
// HEAD_FRAG_ROWS), the same values in the operand order above.  Split-K
// partials still pending from the last layer's down projection (pend->split >
// 0, partials [S, B*L, d]) are added to the head rows of h first, as the fused
// residual norm does; the other rows of h are left without them.  A non-null
// ticket (the LM head's) is set to zero for the head kernel that follows.
void launch_rmsnorm_head(float* h, const PendingResid* pend, const bf16_t* g, bf16_t* out, bf16_t* outf, int B,
                         int rows, int L, int row0, int d, float eps, int* ticket, hipStream_t s);
size_t head_bf16_packed_bytes(int V, int d);
void launch_pack_head_bf16(const bf16_t* W, bf16_t* Wt, int V, int d, hipStream_t s);

struct HeadArgs {
  const bf16_t* hb;   // [R, d]
  const bf16_t* hbf;  // R <= HEAD_FRAG_ROWS: the same rows in MFMA operand order (launch_rmsnorm_head)
  const bf16_t* W;    // tiled copy of the [V, d] LM head (launch_pack_head_bf16)
  int R, V, d, mask_id;
  float* conf; int32_t* argmax; float* logits;  // logits optional
  float* part_m; float* part_s; int32_t* part_i;  // [head_bf16_tiles(V), R]: one slot per workgroup
  int* ticket;                                    // zero before the first launch; left zero
};
void launch_head_bf16(const HeadArgs& a, hipStream_t s);
int head_bf16_tiles(int V);
int head_bf16_max_rows();

// ---- controller (k_commit.hip) ---------------------------------------------
struct CommitArgs {
  int32_t* x; int32_t* commit_step; int8_t* reason; float* sv; int32_t* budget; int32_t* ell; int32_t* done;
  const float* conf; const int32_t* argmax; int32_t* all_done;
  int B, L, P, G, bl, g0, t, T, mask_id;
  float thr[4];        // theta_i(t) per position band (float32)
  int edge[3];         // band edges
  int budget_on, grind_on;
  float s_easy, s_hard; int p_easy, p_hard, b_easy, b_mid, b_hard;
  double eta_bar; int patience; float theta_fb;
  int fixed;           // fixed-schedule baseline instead of the confidence-aware rule
  int fixed_k;         // fixed schedule: tokens to commit this step (0 at steps past the block length)
  // error word of the step's workspace (optional): its bits are reported in
  // *all_done above bit 0 and the word is cleared
  int* err;
  // optional word in coherent pinned host memory: receives seq << 8 | the
  // *all_done value with a system-scope release, so the host can wait for the
  // step by polling it instead of a stream synchronisation
  int* host_flag;
  int seq;
};
void launch_commit(const CommitArgs& a, hipStream_t s);

}  // namespace dllm
