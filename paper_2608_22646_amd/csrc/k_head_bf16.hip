// Fused LM head + vocabulary reduction (Box 1 confidence, greedy prediction).
//
// For each head row r (current block positions of every sequence):
//   logit_v = hb[r, :] . W[v, :]                 (bf16 operands, fp32 accumulate)
//   m = max_{v != mask} logit_v,  s = sum_{v != mask} exp(logit_v - m)
//   conf[r] = 1 / s,  argmax[r] = lowest v != mask with logit_v = m
// The logits never leave registers (unless a debug buffer is given).
//
// Workgroup = 4 wavefronts = 128 vocabulary rows; wave w owns 32 of them and
// every head row (row groups of 32, up to 8).  Per 64-wide k slice a lane
// loads 64 contiguous bytes of one W row (the A operand of four MFMAs) and the
// matching 64 bytes of a head row (the B operand); the k order inside the
// slice is permuted identically on both sides, so the products are unchanged.
// The result layout gives each lane 16 vocabulary entries of one head row,
// merged with lane ^ 32, then across the four waves in order, into one
// (max, sum, argmax) partial per (vocab tile, row).  The last workgroup to
// finish (atomic ticket) merges the partials of all tiles in tile order, so
// the result is independent of scheduling; it then resets the ticket.
#include "kernels.h"

namespace dllm {

namespace {

constexpr int NT = 256, VT = 128;
constexpr float LOG2E = 1.4426950408889634f;

struct Stat {
  float m, s;
  int i;
};

// merge b into a: larger max wins, equal maxima keep the lower index
__device__ __forceinline__ Stat merge(Stat a, Stat b) {
  Stat o;
  o.m = fmaxf(a.m, b.m);
  if (o.m == -INFINITY) {
    o.s = 0.f;
    o.i = min(a.i, b.i);
    return o;
  }
  o.s = a.s * exp2f((a.m - o.m) * LOG2E) + b.s * exp2f((b.m - o.m) * LOG2E);
  o.i = a.m > b.m ? a.i : (b.m > a.m ? b.i : min(a.i, b.i));
  return o;
}

template <int RG>
__global__ void __launch_bounds__(NT, 2) head_bf16_kernel(HeadArgs a) {
  __shared__ Stat wst[4][32 * RG];
  __shared__ int last_flag;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, half = lane >> 5;
  const int v0 = blockIdx.x * VT + wave * 32;
  const int vrow = min(v0 + lr, a.V - 1);
  const bf16_t* wp = a.W + (size_t)vrow * a.d + half * 32;
  const bf16_t* hp[RG];
  bool hval[RG];
#pragma unroll
  for (int g = 0; g < RG; ++g) {
    const int r = g * 32 + lr;
    hval[g] = r < a.R;
    hp[g] = a.hb + (size_t)(hval[g] ? r : 0) * a.d + half * 32;
  }

  f32x16_t acc[RG];
#pragma unroll
  for (int g = 0; g < RG; ++g)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[g][r] = 0.f;

  const int nk = a.d / 64;
  bf16x8_t wc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) wc[j] = *reinterpret_cast<const bf16x8_t*>(wp + j * 8);
  for (int kt = 0; kt < nk; ++kt) {
    bf16x8_t wn[4];
    if (kt + 1 < nk) {
#pragma unroll
      for (int j = 0; j < 4; ++j) wn[j] = *reinterpret_cast<const bf16x8_t*>(wp + (kt + 1) * 64 + j * 8);
    }
#pragma unroll
    for (int g = 0; g < RG; ++g) {
      bf16x8_t hf[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        hf[j] = *reinterpret_cast<const bf16x8_t*>(hp[g] + kt * 64 + j * 8);
        if (!hval[g]) hf[j] = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wc[j], hf[j], acc[g], 0, 0, 0);
    }
    if (kt + 1 < nk) {
#pragma unroll
      for (int j = 0; j < 4; ++j) wc[j] = wn[j];
    }
  }

  // lane holds row g*32 + lr and vocab v0 + 8*(r/4) + 4*half + r%4
#pragma unroll
  for (int g = 0; g < RG; ++g) {
    const int row = g * 32 + lr;
    Stat st{-INFINITY, 0.f, 0x7fffffff};
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int v = v0 + 8 * (r >> 2) + 4 * half + (r & 3);
      const float x = acc[g][r];
      if (a.logits && row < a.R && v < a.V) a.logits[(size_t)row * a.V + v] = x;
      const bool ok = v < a.V && v != a.mask_id;
      if (ok && x > st.m) {
        st.m = x;
        st.i = v;
      }
    }
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int v = v0 + 8 * (r >> 2) + 4 * half + (r & 3);
      if (v < a.V && v != a.mask_id && st.m != -INFINITY) s += exp2f((acc[g][r] - st.m) * LOG2E);
    }
    st.s = s;
    Stat other;
    other.m = __shfl_xor(st.m, 32, 64);
    other.s = __shfl_xor(st.s, 32, 64);
    other.i = __shfl_xor(st.i, 32, 64);
    st = half == 0 ? merge(st, other) : merge(other, st);
    if (half == 0) wst[wave][row] = st;
  }
  __syncthreads();

  // merge the four waves (vocab order) -> tile partial per row
  const int tiles = gridDim.x;
  for (int row = tid; row < a.R; row += NT) {
    Stat st = wst[0][row];
#pragma unroll
    for (int w = 1; w < 4; ++w) st = merge(st, wst[w][row]);
    const size_t o = (size_t)blockIdx.x * a.R + row;
    a.part_m[o] = st.m;
    a.part_s[o] = st.s;
    a.part_i[o] = st.i;
  }
  __threadfence();
  __syncthreads();
  if (tid == 0) last_flag = atomicAdd(a.ticket, 1) == tiles - 1;
  __syncthreads();
  if (!last_flag) return;
  __threadfence();

  // last workgroup: merge tiles in order
  for (int row = tid; row < a.R; row += NT) {
    Stat st{-INFINITY, 0.f, 0x7fffffff};
    for (int t = 0; t < tiles; ++t) {
      const size_t o = (size_t)t * a.R + row;
      Stat p;
      p.m = __builtin_nontemporal_load(a.part_m + o);
      p.s = __builtin_nontemporal_load(a.part_s + o);
      p.i = __builtin_nontemporal_load(a.part_i + o);
      st = merge(st, p);
    }
    a.conf[row] = 1.0f / st.s;
    a.argmax[row] = st.i;
  }
  if (tid == 0) *a.ticket = 0;
}

}  // namespace

int head_bf16_tiles(int V) { return (V + VT - 1) / VT; }
int head_bf16_max_rows() { return 256; }

void launch_head_bf16(const HeadArgs& a, hipStream_t s) {
  if (a.R == 0) return;
  if (a.d % 64 != 0) throw HipError("head_bf16: d % 64 must be 0");
  const dim3 grid(head_bf16_tiles(a.V)), block(NT);
  const int rg = (a.R + 31) / 32;
  if (rg <= 1) hipLaunchKernelGGL(head_bf16_kernel<1>, grid, block, 0, s, a);
  else if (rg <= 2) hipLaunchKernelGGL(head_bf16_kernel<2>, grid, block, 0, s, a);
  else if (rg <= 4) hipLaunchKernelGGL(head_bf16_kernel<4>, grid, block, 0, s, a);
  else hipLaunchKernelGGL(head_bf16_kernel<8>, grid, block, 0, s, a);
  DLLM_LAUNCH_CHECK("head_bf16");
}

}  // namespace dllm
