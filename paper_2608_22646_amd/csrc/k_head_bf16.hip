// Fused LM head + vocabulary reduction (Box 1 confidence, greedy prediction).
//
// For each head row r (current block positions of every sequence):
//   logit_v = hb[r, :] . W[v, :]                 (bf16 operands, fp32 accumulate)
//   m = max_{v != mask} logit_v,  s = sum_{v != mask} exp(logit_v - m)
//   conf[r] = 1 / s,  argmax[r] = lowest v != mask with logit_v = m
// The logits never leave registers (unless a debug buffer is given); the kernel
// is bound by streaming W (V x d bf16) from HBM once.
//
// W is read from a tiled copy made once per model: for vocabulary tile t of
// HEAD_TILE rows and k-block kb of 64, the [HEAD_TILE, 64] block is stored
// contiguously, blocks in (t, kb) order.  A ring slice (VT rows x 64 k) is then
// one contiguous 16-32 KB run of HBM: streaming 128-byte pieces of hundreds of
// rows 8 KB apart instead reaches only about 70% of the contiguous rate.
//
// Persistent grid: G workgroups (one or two per CU) walk vocabulary tiles of
// VT = 32 NW rows (NW waves), tile = blockIdx.x + i*G.  The tiles' (tile,
// k-step of 64) slices stream through an S-stage LDS ring filled by
// buffer_load_dwordx4 ... lds (whole 128-byte lines per eight lanes),
// continuing across tile boundaries, so S-1 slices are always in flight; the
// ring depth and tile height are chosen per head-row count so that W is most of
// each slice (the hb rows ride along) and the ring fills the CU's LDS.  Wave w
// owns 32 vocabulary rows of the tile and every head row (groups of 32):
// A = W rows, B = hb rows of the MFMA, so a lane ends up with 16 vocabulary
// entries of one head row.  Per tile those are merged across the lane pair and
// the waves into a per-row running
// (max, sum, argmax) that thread r keeps in registers over all of the
// workgroup's tiles.  At the end each workgroup publishes one partial per row
// (device-coherent sc1 stores, no cache flush); the last workgroup to finish
// (atomic ticket) merges the G partials in workgroup order, so the result is
// independent of scheduling, writes conf / argmax and re-arms the ticket.
#include "kernels.h"

namespace dllm {

namespace {

constexpr int BK = 64;
constexpr int MAX_WG = 512;  // partial slots per row in the workspace
constexpr float LOG2E = 1.4426950408889634f;
constexpr int CPOL_SC1 = 16;  // cache-policy bit: coherent at device (agent) scope

typedef __attribute__((address_space(3))) void* lds_ptr_t;

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

// wait until at most N vector-memory operations of this wave are outstanding
// and all of its LDS operations are done (s_waitcnt vmcnt(N) lgkmcnt(0))
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void barrier_nofence_h() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
// 16-byte chunk c of 128-byte LDS row r lives in slot c ^ ((r >> 1) & 7): the
// 16 consecutive rows that one 16-lane pass of ds_read_b128 touches then cover
// all 64 banks (two rows per 256-byte bank line, eight slots each).
__device__ __forceinline__ int swz(int row, int chunk) { return row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4); }

template <int RG, int VT, int NW, int S>
__global__ void __launch_bounds__(64 * NW, 1) head_bf16_kernel(HeadArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  static_assert(VT == 32 * NW && S >= 3 && HEAD_TILE % VT == 0, "tile shape");
  constexpr int NT = 64 * NW;
  constexpr int HR = 32 * RG;                           // head rows covered
  constexpr int STAGE = (VT + HR) * 128;                // W slice + hb slice
  constexpr int IW = VT / 8 / NW;                       // W DMA instructions per wave per slice
  constexpr int HQ = HR / 8;                            // hb DMA instructions per slice, spread over waves
  constexpr int IH_HI = (HQ + NW - 1) / NW, IH_LO = HQ / NW;
  extern __shared__ __attribute__((aligned(16))) char lds[];
  __shared__ Stat wst[NW][HR];
  __shared__ int last_flag;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool hb_hi = HQ % NW == 0 || wave < HQ % NW;   // this wave issues IH_HI hb loads per slice
  const int lr = lane & 31, half = lane >> 5;
  const int G = gridDim.x;
  const int ntiles = (a.V + HEAD_TILE - 1) / HEAD_TILE * (HEAD_TILE / VT);
  const int nk = a.d / BK;
  const int my_tiles = blockIdx.x < ntiles ? (ntiles - 1 - blockIdx.x) / G + 1 : 0;
  const int units = my_tiles * nk;

  // DMA sources: instruction i of wave w fills rows 8 (NW i + w) .. +7 of the
  // slice; lane l loads row + l/8, logical chunk (l%8) ^ ((row >> 1) & 7) into
  // slot l%8 (NW even: row >> 1 = 4 (w & 1) + (l/8) / 2 modulo 8 for every i).
  const int dr = lane >> 3, dc = (lane & 7) ^ (((wave & 1) << 2) | (dr >> 1));
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc((void*)a.hb, 0, 0x7fffffff, 0x00020000);
  uint32_t voh[IH_HI];
#pragma unroll
  for (int i = 0; i < IH_HI; ++i) {
    const int row = min(8 * (NW * i + wave) + dr, a.R - 1);
    voh[i] = (uint32_t)(((size_t)row * a.d + dc * 8) * 2);
  }
  auto issue = [&](int u) {
    const int tile = blockIdx.x + (u / nk) * G, kk = u % nk;
    char* base = lds + (u % S) * STAGE;
#pragma unroll
    for (int i = 0; i < IW; ++i) {
      const int lt = tile / (HEAD_TILE / VT), r0 = (tile % (HEAD_TILE / VT)) * VT;
      const int row = r0 + 8 * (NW * i + wave) + dr;  // row within the layout tile
      const uint32_t vo = (uint32_t)((((size_t)lt * nk + kk) * HEAD_TILE + row) * 128 + dc * 16);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)(base + 8 * (NW * i + wave) * 128), 16, vo, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < IH_HI; ++i)
      if (i < IH_LO || hb_hi)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rh, (lds_ptr_t)(base + VT * 128 + 8 * (NW * i + wave) * 128), 16,
                                                 voh[i] + kk * BK * 2, 0, 0, 0);
  };

  Stat run{-INFINITY, 0.f, 0x7fffffff};  // thread r < R: running stats of head row r
  f32x16_t acc[RG];
#pragma unroll
  for (int s = 0; s < S - 1; ++s)
    if (s < units) issue(s);

  for (int u = 0; u < units; ++u) {
    const int kk = u % nk;
    if (kk == 0) {
#pragma unroll
      for (int gi = 0; gi < RG; ++gi)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[gi][r] = 0.f;
    }
    // this wave's loads for unit u are done once at most the S-2 later units'
    // loads are outstanding (loads complete in order)
    if (u + S - 2 >= units)
      wait_vm_lds<0>();  // (only reached near the end: fewer later units were issued)
    else if (hb_hi)
      wait_vm_lds<(IW + IH_HI) * (S - 2)>();
    else
      wait_vm_lds<(IW + IH_LO) * (S - 2)>();
    barrier_nofence_h();
    if (u + S - 1 < units) issue(u + S - 1);
    const char* base = lds + (u % S) * STAGE;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = ks * 2 + half;
      const bf16x8_t wf = *reinterpret_cast<const bf16x8_t*>(base + swz(wave * 32 + lr, ch));
#pragma unroll
      for (int gi = 0; gi < RG; ++gi) {
        const bf16x8_t hf = *reinterpret_cast<const bf16x8_t*>(base + VT * 128 + swz(gi * 32 + lr, ch));
        acc[gi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf, hf, acc[gi], 0, 0, 0);
      }
    }
    if (kk != nk - 1) continue;

    // ---- tile epilogue: lane holds head row gi*32 + lr, vocab v0 + 8(r/4) + 4 half + r%4
    const int tile = blockIdx.x + (u / nk) * G;
    const int v0 = tile * VT + wave * 32;
#pragma unroll
    for (int gi = 0; gi < RG; ++gi) {
      const int row = gi * 32 + lr;
      Stat st{-INFINITY, 0.f, 0x7fffffff};
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = v0 + 8 * (r >> 2) + 4 * half + (r & 3);
        const float x = acc[gi][r];
        if (a.logits && row < a.R && v < a.V) a.logits[(size_t)row * a.V + v] = x;
        if (v < a.V && v != a.mask_id && x > st.m) {
          st.m = x;
          st.i = v;
        }
      }
      float s = 0.f;
      if (st.m != -INFINITY) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = v0 + 8 * (r >> 2) + 4 * half + (r & 3);
          if (v < a.V && v != a.mask_id) s += exp2f((acc[gi][r] - st.m) * LOG2E);
        }
      }
      st.s = s;
      Stat other;
      other.m = __shfl_xor(st.m, 32, 64);
      other.s = __shfl_xor(st.s, 32, 64);
      other.i = __shfl_xor(st.i, 32, 64);
      st = half == 0 ? merge(st, other) : merge(other, st);
      if (half == 0) wst[wave][row] = st;
    }
    // LDS barrier that leaves the ring's DMA in flight (__syncthreads would
    // wait for it); wst is next written after the following unit's barrier
    wait_vm_lds<63>();
    barrier_nofence_h();
    if (tid < a.R) {
      Stat st = wst[0][tid];
#pragma unroll
      for (int w = 1; w < NW; ++w) st = merge(st, wst[w][tid]);
      run = merge(run, st);
    }
  }

  // ---- publish this workgroup's partial per row, then the last one merges
  const __amdgpu_buffer_rsrc_t rm = __builtin_amdgcn_make_buffer_rsrc((void*)a.part_m, 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void*)a.part_s, 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ri = __builtin_amdgcn_make_buffer_rsrc((void*)a.part_i, 0, 0x7fffffff, 0x00020000);
  if (tid < a.R) {
    const uint32_t off = (uint32_t)(((size_t)blockIdx.x * a.R + tid) * 4);
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(run.m), rm, off, 0, CPOL_SC1);
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(run.s), rs, off, 0, CPOL_SC1);
    __builtin_amdgcn_raw_buffer_store_b32((uint32_t)run.i, ri, off, 0, CPOL_SC1);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) last_flag = atomicAdd(a.ticket, 1) == G - 1;
  __syncthreads();
  if (!last_flag) return;

  // last workgroup: TPR threads per row merge strided runs of the G partials,
  // then the runs are combined in order; both orders are fixed.  The loads of
  // a run are issued 16 at a time so their latencies overlap.
  constexpr int TPR_MAX = 8, LB = 16;
  const int tpr = a.R <= NT / TPR_MAX ? TPR_MAX : (a.R <= NT / 4 ? 4 : (a.R <= NT / 2 ? 2 : 1));
  Stat* fin = reinterpret_cast<Stat*>(lds);  // the ring is idle now
  const int row = tid / tpr, sub = tid % tpr;
  Stat st{-INFINITY, 0.f, 0x7fffffff};
  if (row < a.R) {
    for (int g0 = sub; g0 < G; g0 += LB * tpr) {
      Stat p[LB];
#pragma unroll
      for (int j = 0; j < LB; ++j) {
        const int gwg = min(g0 + j * tpr, G - 1);
        const uint32_t off = (uint32_t)(((size_t)gwg * a.R + row) * 4);
        p[j].m = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rm, off, 0, CPOL_SC1));
        p[j].s = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, CPOL_SC1));
        p[j].i = (int)__builtin_amdgcn_raw_buffer_load_b32(ri, off, 0, CPOL_SC1);
      }
#pragma unroll
      for (int j = 0; j < LB; ++j)
        if (g0 + j * tpr < G) st = merge(st, p[j]);
    }
  }
  fin[tid] = st;
  __syncthreads();
  if (row < a.R && sub == 0) {
    Stat t = fin[tid];
    for (int j = 1; j < tpr; ++j) t = merge(t, fin[tid + j]);
    a.conf[row] = 1.0f / t.s;
    a.argmax[row] = t.i;
  }
  if (tid == 0) *a.ticket = 0;
#endif
}

// one thread per 16-byte vector of the tiled copy, in destination order
__global__ void pack_head_kernel(const bf16_t* __restrict__ W, bf16_t* __restrict__ Wt, int V, int d, size_t nvec) {
  const int nk = d / 64;
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < nvec; idx += (size_t)gridDim.x * blockDim.x) {
    const int c8 = (int)(idx % 8);
    size_t t = idx / 8;
    const int r = (int)(t % HEAD_TILE);
    t /= HEAD_TILE;
    const int kb = (int)(t % nk);
    const size_t lt = t / nk;
    const size_t row = lt * HEAD_TILE + r;
    bf16x8_t v = {};
    if (row < (size_t)V) v = *reinterpret_cast<const bf16x8_t*>(W + row * d + kb * 64 + c8 * 8);
    *reinterpret_cast<bf16x8_t*>(Wt + idx * 8) = v;
  }
}


// one launch shape: RG groups of 32 head rows, vocabulary tiles of VT rows on
// NW waves, an S-stage ring
template <int RG, int VT, int NW, int S>
struct HeadCfg {
  static constexpr int HR = 32 * RG;
  static constexpr size_t lds = (size_t)S * (VT + HR) * 128;
  static constexpr size_t lds_all = lds + NW * HR * sizeof(Stat) + 16;
  static_assert(lds_all <= 160 * 1024, "LDS budget");
  static_assert(lds >= 64 * NW * sizeof(Stat), "final merge staging lives in the ring");
  static int ntiles(int V) { return (V + HEAD_TILE - 1) / HEAD_TILE * (HEAD_TILE / VT); }
  static int grid(int V) {
    const int per_cu = 2 * lds_all <= 160 * 1024 ? 2 : 1;
    return std::min(std::min(ntiles(V), device_cu_count() * per_cu), MAX_WG);
  }
  static void launch(const HeadArgs& a, hipStream_t s) {
    static const hipError_t attr = hipFuncSetAttribute((const void*)head_bf16_kernel<RG, VT, NW, S>,
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hip_check(attr, "hipFuncSetAttribute(head_bf16)");
    hipLaunchKernelGGL((head_bf16_kernel<RG, VT, NW, S>), dim3(grid(a.V)), dim3(64 * NW), lds, s, a);
  }
};

}  // namespace

size_t head_bf16_packed_bytes(int V, int d) {
  return (size_t)ceil_div(V, HEAD_TILE) * HEAD_TILE * (size_t)d * sizeof(bf16_t);
}

void launch_pack_head_bf16(const bf16_t* W, bf16_t* Wt, int V, int d, hipStream_t s) {
  if (d % 64 != 0) throw HipError("pack_head: d % 64 must be 0");
  const size_t nvec = head_bf16_packed_bytes(V, d) / 16;
  const int grid = (int)std::min<size_t>(ceil_div(nvec, (size_t)256), 8192);
  hipLaunchKernelGGL(pack_head_kernel, dim3(grid), dim3(256), 0, s, W, Wt, V, d, nvec);
  DLLM_LAUNCH_CHECK("pack_head_bf16");
}

int head_bf16_tiles(int) { return MAX_WG; }  // partial slots: one per workgroup
int head_bf16_max_rows() { return 256; }

void launch_head_bf16(const HeadArgs& a, hipStream_t s) {
  if (a.R == 0) return;
  if (a.d % BK != 0) throw HipError("head_bf16: d % 64 must be 0");
  if (head_bf16_packed_bytes(a.V, a.d) > 0x7fffffffu) throw HipError("head_bf16: LM head larger than 2 GiB");
  const int rg = (a.R + 31) / 32;
  // (head-row groups, vocab tile, waves, ring stages).  Eight waves per CU
  // stream faster than four whatever the ring depth, so 256-row tiles are kept
  // even where the tile count divides unevenly over the CUs.
  if (rg <= 1) HeadCfg<1, 256, 8, 4>::launch(a, s);
  else if (rg <= 2) HeadCfg<2, 256, 8, 3>::launch(a, s);
  else if (rg <= 4) HeadCfg<4, 128, 4, 3>::launch(a, s);
  else HeadCfg<8, 128, 4, 3>::launch(a, s);
  DLLM_LAUNCH_CHECK("head_bf16");
}

}  // namespace dllm
