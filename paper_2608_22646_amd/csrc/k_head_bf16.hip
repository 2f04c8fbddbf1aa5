// Fused LM head + vocabulary reduction (Box 1 confidence, greedy prediction).
//
// For each head row r (current block positions of every sequence):
//   logit_v = hb[r, :] . W[v, :]                 (bf16 operands, fp32 accumulate)
//   m = max_{v != mask} logit_v,  s = sum_{v != mask} exp(logit_v - m)
//   conf[r] = 1 / s,  argmax[r] = lowest v != mask with logit_v = m
// The logits never leave registers (unless a debug buffer is given); the kernel
// is bound by streaming W (V x d bf16) from HBM once.
//
// W is read from a tiled copy made once per model, in MFMA fragment order: for
// vocabulary tile t of HEAD_TILE rows and k-block kb of 64, the [HEAD_TILE, 64]
// block is stored contiguously (blocks in (t, kb) order), and inside it each
// 32-row x 16-k operand of v_mfma_f32_32x32x16_bf16 is one 1 KiB run in lane
// order (group of 32 rows g, then k-slice s, then lane l = row % 32 + 32 *
// (8-column half), 16 bytes per lane).  A (tile, 64-k) slice is then one
// contiguous run of HBM, and a wave's A operand is one 1 KiB load.
//
// Two kernels share that layout and the final merge:
//  * head_stream_kernel (up to 32 head rows): every wave streams the 1 KiB
//    operands of its own 32 vocabulary rows straight into registers, P slices
//    in flight, with no LDS ring and no barrier in the loop; the head rows'
//    operands come from the (cache-resident) hb rows alongside.
//  * head_bf16_kernel (more head rows): the tiles' (tile, k-step of 64)
//    slices stream through an S-stage LDS ring filled by buffer_load_dwordx4
//    ... lds, continuing across tile boundaries, so S-1 slices are always in
//    flight; the ring depth and tile height are chosen per head-row count so
//    that W is most of each slice (the hb rows ride along, row-major and
//    swizzled) and the ring fills the CU's LDS.
// In both, persistent workgroups walk vocabulary tiles (tile = blockIdx.x +
// i*G); wave w owns 32 vocabulary rows of the tile and every head row (groups
// of 32): A = W rows, B = hb rows of the MFMA, so a lane ends up with 16
// vocabulary entries of one head row.  Per tile those are merged across the
// lane pair into per-row running (max, sum, argmax) statistics.  At the end
// each workgroup publishes one partial per row (device-coherent sc1 stores,
// no cache flush); the last workgroup to finish (atomic ticket) merges the G
// partials in workgroup order, so the result is independent of scheduling,
// writes conf / argmax and re-arms the ticket.
#include "kernels.h"

namespace dllm {

namespace {

constexpr int BK = 64;
constexpr int MAX_WG = 512;  // partial slots per row in the workspace
constexpr float LOG2E = 1.4426950408889634f;
constexpr int CPOL_SC1 = 16;  // cache-policy bit: coherent at device (agent) scope
constexpr int CPOL_NT = 2;    // cache-policy bit: non-temporal (W is streamed once)

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

// Bytes of the tiled copy (head_bf16_packed_bytes), device side.
__device__ __forceinline__ size_t head_bf16_packed_bytes_dev(int V, int d) {
  return (size_t)((V + HEAD_TILE - 1) / HEAD_TILE) * HEAD_TILE * (size_t)d * 2;
}

// Statistics of one 32-row vocabulary group for head row `row` from the MFMA
// result (lane holds vocabulary entries v0 + 8 (r/4) + 4 half + r%4, r < 16),
// merged across the lane pair: valid in the half == 0 lane.  Writes the logits
// too when a debug buffer is given.
template <bool LG = true>
__device__ __forceinline__ Stat tile_stat(const HeadArgs& a, const f32x16_t& acc, int row, int v0, int half) {
  Stat st{-INFINITY, 0.f, 0x7fffffff};
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int v = v0 + 8 * (r >> 2) + 4 * half + (r & 3);
    const float x = acc[r];
    if (LG && a.logits && row < a.R && v < a.V) a.logits[(size_t)row * a.V + v] = x;
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
      if (v < a.V && v != a.mask_id) s += exp2f((acc[r] - st.m) * LOG2E);
    }
  }
  st.s = s;
  Stat other;
  other.m = __shfl_xor(st.m, 32, 64);
  other.s = __shfl_xor(st.s, 32, 64);
  other.i = __shfl_xor(st.i, 32, 64);
  return half == 0 ? merge(st, other) : merge(other, st);
}

// Thread tid < R holds this workgroup's statistics of head row tid.  Publishes
// them (one partial per (workgroup, row), device-coherent sc1 stores), takes a
// ticket, and the last workgroup merges the G partials of every row in
// workgroup order and writes conf / argmax.  fin: NT Stats of idle LDS.
template <int NT>
__device__ __forceinline__ void publish_and_merge(const HeadArgs& a, const Stat& run, int tid, Stat* fin,
                                                  int& last_flag) {
  const int G = gridDim.x;
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
}

template <int RG, int VT, int NW, int S>
__global__ void __launch_bounds__(64 * NW, 1) head_bf16_kernel(HeadArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  static_assert(VT == 32 * NW && S >= 3 && HEAD_TILE % VT == 0 && VT / 8 / NW == 4, "tile shape");
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

  // DMA sources: W instruction i of wave w copies the 1 KiB operand block
  // j = NW i + w of the slice (group j / 4, k-slice j % 4) to LDS offset j KiB.
  // hb instruction i of wave w fills rows 8 (NW i + w) .. +7 of the hb part;
  // lane l loads row + l/8, logical chunk (l%8) ^ ((row >> 1) & 7) into slot
  // l%8 (NW even: row >> 1 = 4 (w & 1) + (l/8) / 2 modulo 8 for every i).
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
      const int lt = tile / (HEAD_TILE / VT), g0 = (tile % (HEAD_TILE / VT)) * (VT / 32);
      const int j = NW * i + wave;
      const uint32_t vo =
          (uint32_t)((((size_t)lt * nk + kk) * HEAD_TILE * 128) + ((size_t)g0 * 4 + j) * 1024 + lane * 16);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)(base + j * 1024), 16, vo, 0, 0, CPOL_NT);
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
      const bf16x8_t wf = *reinterpret_cast<const bf16x8_t*>(base + ((4 * wave + ks) * 64 + lane) * 16);
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
      const Stat st = tile_stat(a, acc[gi], gi * 32 + lr, v0, half);
      if (half == 0) wst[wave][gi * 32 + lr] = st;
    }
    // debug logits stores count in vmcnt too: drain them so the ring's counts
    // keep describing its loads only
    if (a.logits) wait_vm_lds<0>();
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

  publish_and_merge<NT>(a, run, tid, reinterpret_cast<Stat*>(lds), last_flag);
#endif
}

// Streaming kernel for up to 32 head rows: NW = 4 waves per workgroup, one
// per SIMD; a workgroup tile is 32 GW NW vocabulary rows and wave w owns its GW
// groups w GW .. w GW + GW - 1 of 32 rows (each group lies inside one tile of
// the copy, so any GW works).  The wave walks the tiles' 16-k
// slices in order; per slice it loads the GW 1 KiB W operands and the 1 KiB hb
// operand (the operand-order copy) into a P-deep register ring, so one hb load
// serves GW MFMAs.  Loads complete in issue order, so before slice u only the
// (GW + 1) (P - 1) loads of the slices after it may be outstanding.  W reads
// past the tiled copy (a last tile that extends beyond it) return zeros
// through the buffer bound.
template <int GW, int P>
__global__ void __launch_bounds__(256, 1) head_stream_kernel(HeadArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int NW = 4, NT = 64 * NW, TROWS = 32 * GW * NW;
  static_assert(HEAD_TILE % 32 == 0 && (GW + 1) * (P - 1) < 64, "tile shape");
  __shared__ Stat wst[NW][32];
  __shared__ Stat fin[NT];
  __shared__ int last_flag;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 31, half = lane >> 5;
  const int G = gridDim.x;
  const int ntiles = (a.V + TROWS - 1) / TROWS;
  const int nk = a.d / BK, ns = 4 * nk;
  const int my_tiles = blockIdx.x < ntiles ? (ntiles - 1 - blockIdx.x) / G + 1 : 0;
  const int units = my_tiles * ns;

  const uint32_t wbytes = (uint32_t)head_bf16_packed_bytes_dev(a.V, a.d);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, 0, wbytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc((void*)a.hbf, 0, 0x7fffffff, 0x00020000);
  // first vocabulary row of group j of this wave in tile t: t TROWS + (wave GW + j) 32;
  // in the copy: layout tile r / HEAD_TILE, group (r % HEAD_TILE) / 32
  typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
  u32x4_t wbuf[P][GW], hbuf[P];
  auto load = [&](int u, int slot) {
    const int t = blockIdx.x + (u / ns) * G, sl = u % ns;
#pragma unroll
    for (int j = 0; j < GW; ++j) {
      const int r0 = t * TROWS + (wave * GW + j) * 32;
      const int lt = r0 / HEAD_TILE, g8 = (r0 % HEAD_TILE) / 32;
      const uint32_t wo =
          (uint32_t)((((size_t)lt * nk + (sl >> 2)) * (HEAD_TILE / 32) + g8) * 4 + (sl & 3)) * 1024 + lane * 16;
      wbuf[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(rw, wo, 0, CPOL_NT);
    }
    hbuf[slot] = __builtin_amdgcn_raw_buffer_load_b128(rh, (uint32_t)(sl * 1024 + lane * 16), 0, 0);
  };
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (p < units) load(p, p);

  Stat run{-INFINITY, 0.f, 0x7fffffff};  // lane lr (half 0): running stats of head row lr
  f32x16_t acc[GW];
#pragma unroll
  for (int j = 0; j < GW; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  // ns is a multiple of P (the launcher checks d % (16 P) == 0), so slice u sits
  // in ring slot u % P = p
  for (int ti = 0; ti < my_tiles; ++ti) {
    for (int s0 = 0; s0 < ns; s0 += P) {
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const int u = ti * ns + s0 + p;
        if (u + P - 1 < units)
          wait_vm_lds<(GW + 1) * (P - 1)>();
        else
          wait_vm_lds<0>();  // the last slices: fewer later loads were issued
#pragma unroll
        for (int j = 0; j < GW; ++j)
          acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wbuf[p][j]),
                                                          __builtin_bit_cast(bf16x8_t, hbuf[p]), acc[j], 0, 0, 0);
        if (u + P < units) load(u + P, p);
      }
    }
    // end of a tile: this wave's vocabulary rows are complete
    const int t = blockIdx.x + ti * G;
#pragma unroll
    for (int j = 0; j < GW; ++j) {
      const Stat st = tile_stat(a, acc[j], lr, t * TROWS + (wave * GW + j) * 32, half);
      run = merge(run, st);
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
    }
    // debug logits stores count in vmcnt too: drain them so the counts above
    // keep describing loads only
    if (a.logits) wait_vm_lds<0>();
  }
  if (half == 0) wst[wave][lr] = run;
  __syncthreads();
  Stat wg{-INFINITY, 0.f, 0x7fffffff};
  if (tid < a.R) {
    wg = wst[0][tid];
#pragma unroll
    for (int w = 1; w < NW; ++w) wg = merge(wg, wst[w][tid]);
  }
  publish_and_merge<NT>(a, wg, tid, fin, last_flag);
#endif
}

// Register-direct variant for more than 32 head rows (batched decodes): the
// workgroup tile is one 256-row vocabulary tile of the copy x all head rows
// (up to 32 TI); wave w owns the tile's 32-row groups 2w and 2w + 1, whose
// 1 KiB operands stream straight from the copy into a register ring of P slices
// (non-temporal; four slices at 256 head rows, where the accumulators fill the
// AGPRs), while the head rows' 64-k slice of each k-step is staged by LDS-DMA
// in a 4-stage ring (one barrier per k-step) that all four waves read.
// In the LDS-ring kernel above every wave re-reads all head rows from LDS for
// its 32 vocabulary rows; here each head-row fragment serves two MFMAs and the
// vocabulary rows never touch LDS.  Per slice a wave runs 2 TI MFMAs with W as
// the A operand; at the end of a tile the lanes' entries are reduced
// (tile_stat), merged across the waves through LDS into the per-row running
// statistics, and the workgroups' partials merged as in the other kernels.
// The ring's issue order and wait counts are those of the register-direct GEMM
// (stages of one 64-k step: four slices per stage, two DMA loads per slice).
template <int TI, bool LG>
__global__ void __launch_bounds__(256, 1) head_wd_kernel(HeadArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  // a 4-slice weight ring at 256 head rows, where the accumulators fill the AGPRs
  constexpr int NW = 4, NT = 256, TJ = 2, AS = 4, P = TI == 8 ? 4 : 8, U = 4, BM = 32 * TI, R2 = P / U;
  constexpr int STAGE = BM * 128;   // head rows x 64 k
  constexpr int IA = BM / 8 / NW;   // DMA loads per wave per stage
  constexpr int IU = IA / U;        // ... per slice
  static_assert(IU * U == IA && IU >= 1 && HEAD_TILE == 32 * TJ * NW, "tile shape");
  constexpr int PER = TJ + IU;
  constexpr int C1 = TJ + (AS - 3) * U * PER + (U - 1) * PER + IU;
  constexpr int C0 = (AS - 3) * IA + P * TJ + (U - 1) * PER + IU;
  constexpr int CMIN = C0 < C1 ? C0 : C1;
  constexpr int CWAIT = CMIN < 63 ? CMIN : 63;
  constexpr int CFIRST = ((AS - 2) * IA + P * TJ) < 63 ? (AS - 2) * IA + P * TJ : 63;
  extern __shared__ __attribute__((aligned(16))) char lds[];
  __shared__ Stat wst[NW][BM];
  __shared__ Stat fin[NT];
  __shared__ int last_flag;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int G = gridDim.x, nk = a.d / BK;
  const int ntiles = (a.V + HEAD_TILE - 1) / HEAD_TILE;
  const int my_tiles = blockIdx.x < ntiles ? (ntiles - 1 - blockIdx.x) / G + 1 : 0;
  const int units = my_tiles * nk;  // stages: (tile, 64-k step)

  // head-row DMA: instruction q of wave w fills rows 8 (4 q + w) .. +7; lane l
  // writes row + l/8, slot l%8 holding chunk (l%8) ^ ((row >> 1) & 7); rows
  // past R repeat the last row (never used)
  const int dr = lane >> 3, dc = (lane & 7) ^ (((wave & 1) << 2) | (dr >> 1));
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc((void*)a.hb, 0, 0x7fffffff, 0x00020000);
  uint32_t voh[IA];
#pragma unroll
  for (int q = 0; q < IA; ++q) {
    const int row = min(8 * (4 * q + wave) + dr, a.R - 1);
    voh[q] = (uint32_t)(((size_t)row * a.d + dc * 8) * 2);
  }
  // stage u's LDS slot and head-row k offset (past the end: the last stage
  // again, never read), and the byte offset of its 32 KiB (tile, k-step) run
  // of the copy; computed once per stage
  auto a_soff = [&](int u) { return (min(u, units - 1) % nk) * BK * 2; };
  auto w_run = [&](int u) {
    u = min(u, units - 1);
    const int i = u / nk;
    return (uint32_t)(((size_t)(blockIdx.x + i * G) * nk + (u - i * nk)) * (HEAD_TILE / 32) * 4 * 1024);
  };
  auto issue_a = [&](int slot, int soff, int q) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rh, (lds_ptr_t)(lds + slot * STAGE + 8 * (4 * q + wave) * 128), 16,
                                             voh[q], soff, 0, 0);
  };
  const uint32_t wbytes = (uint32_t)head_bf16_packed_bytes_dev(a.V, a.d);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, 0, wbytes, 0x00020000);
  typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
  u32x4_t wbuf[P][TJ];
  const uint32_t wlane = (uint32_t)(2 * wave * 4 * 1024 + lane * 16);
  // operand j (group 2 wave + j of the tile) of slice sl of the stage whose run starts at run
  auto load_w = [&](uint32_t run, int sl, int slot, int j) {
    wbuf[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(rw, run + wlane + (uint32_t)((j * 4 + sl) * 1024), 0,
                                                          CPOL_NT);
  };
  bf16x8_t af[2][TI];
  auto frag = [&](const char* base, int sl, int set) {
#pragma unroll
    for (int ii = 0; ii < TI; ++ii)
      af[set][ii] = *reinterpret_cast<const bf16x8_t*>(base + swz(32 * ii + lrow, 2 * sl + lhalf));
  };
  f32x16_t acc[TJ][TI];
#pragma unroll
  for (int j = 0; j < TJ; ++j)
#pragma unroll
    for (int ii = 0; ii < TI; ++ii)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][ii][r] = 0.f;
  Stat run{-INFINITY, 0.f, 0x7fffffff};  // thread r < R: running statistics of head row r

  static_assert(P % U == 0, "slices P later are in stage u + P / U");
  if (units > 0) {
#pragma unroll
    for (int t = 0; t < AS - 1; ++t)
#pragma unroll
      for (int q = 0; q < IA; ++q) issue_a(t, a_soff(t), q);
#pragma unroll
    for (int v = 0; v < P; ++v)
#pragma unroll
      for (int j = 0; j < TJ; ++j) load_w(w_run(v / U), v % U, v, j);
    wait_vm_lds<CFIRST>();
    barrier_nofence_h();
    frag(lds, 0, 0);
  }
  for (int ti = 0; ti < my_tiles; ++ti) {
    for (int k0 = 0; k0 < nk; k0 += R2) {
#pragma unroll
      for (int rr = 0; rr < R2; ++rr) {
        const int u = ti * nk + k0 + rr;
        const char* base = lds + (u % AS) * STAGE;
        // this stage's loads: the DMA of stage u + AS - 1, the weights of stage u + P / U
        const int aslot = (u + AS - 1) % AS, asoff = a_soff(u + AS - 1);
        const uint32_t wnext = w_run(u + P / U);
#pragma unroll
        for (int sl = 0; sl < U; ++sl) {
          const int slot = (rr * U + sl) % P;
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int q = 0; q < IU; ++q) issue_a(aslot, asoff, sl * IU + q);
          if (sl + 1 < U) {
            frag(base, sl + 1, (sl + 1) & 1);
          } else {
            wait_vm_lds<CWAIT>();
            barrier_nofence_h();
            frag(lds + ((u + 1) % AS) * STAGE, 0, 0);
          }
#pragma unroll
          for (int j = 0; j < TJ; ++j) {
#pragma unroll
            for (int ii = 0; ii < TI; ++ii)
              acc[j][ii] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wbuf[slot][j]),
                                                                  af[sl & 1][ii], acc[j][ii], 0, 0, 0);
            load_w(wnext, sl, slot, j);
          }
          __builtin_amdgcn_sched_group_barrier(0x020, IU, 0);
#pragma unroll
          for (int j = 0; j < TJ; ++j) {
            if (j == 0) {
#pragma unroll
              for (int ii = 0; ii < TI; ++ii) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
              }
            } else {
              __builtin_amdgcn_sched_group_barrier(0x008, TI, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
          }
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    // end of a vocabulary tile: lane holds head row 32 ii + lrow, entries
    // v0 + 8 (r / 4) + 4 lhalf + r % 4 of group 2 wave + j
    const int t = blockIdx.x + ti * G;
#pragma unroll
    for (int ii = 0; ii < TI; ++ii) {
      Stat st = tile_stat<LG>(a, acc[0][ii], 32 * ii + lrow, t * HEAD_TILE + (2 * wave) * 32, lhalf);
      st = merge(st, tile_stat<LG>(a, acc[1][ii], 32 * ii + lrow, t * HEAD_TILE + (2 * wave + 1) * 32, lhalf));
      if (lhalf == 0) wst[wave][32 * ii + lrow] = st;
      __builtin_amdgcn_sched_barrier(0);  // one row block at a time (register pressure)
    }
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int ii = 0; ii < TI; ++ii)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][ii][r] = 0.f;
    // debug logits stores count in vmcnt too: drain them so the ring's
    // counts keep describing its loads only
    if (LG) wait_vm_lds<0>();
    // an LDS barrier that leaves the ring's loads in flight; wst is next
    // written a whole tile (and many barriers) later
    wait_vm_lds<63>();
    barrier_nofence_h();
    if (tid < a.R) {
      Stat w = wst[0][tid];
#pragma unroll
      for (int x = 1; x < NW; ++x) w = merge(w, wst[x][tid]);
      run = merge(run, w);
    }
  }
  wait_vm_lds<0>();
  publish_and_merge<NT>(a, run, tid, fin, last_flag);
#endif
}

// one thread per 16-byte vector of the tiled copy, in destination order
__global__ void pack_head_kernel(const bf16_t* __restrict__ W, bf16_t* __restrict__ Wt, int V, int d, size_t nvec) {
  const int nk = d / 64;
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < nvec; idx += (size_t)gridDim.x * blockDim.x) {
    // destination vector idx = ((lt * nk + kb) * 8 + g) * 4 + s) * 64 + l
    const int l = (int)(idx % 64);
    size_t t = idx / 64;
    const int sl = (int)(t % 4);
    t /= 4;
    const int g = (int)(t % (HEAD_TILE / 32));
    t /= HEAD_TILE / 32;
    const int kb = (int)(t % nk);
    const size_t lt = t / nk;
    const size_t row = lt * HEAD_TILE + g * 32 + (l & 31);
    const int k = kb * 64 + sl * 16 + (l >> 5) * 8;
    bf16x8_t v = {};
    if (row < (size_t)V) v = *reinterpret_cast<const bf16x8_t*>(W + row * d + k);
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
  if (a.R <= HEAD_FRAG_ROWS && a.hbf && a.d % 256 == 0) {
    // streaming kernel, one workgroup per CU: the tile height (128, 256, 512 or
    // 640 rows: GW = 1, 2, 4, 5 groups per wave) that minimises the largest
    // number of rows a CU streams, weighted by the hb loads per W load (1 / GW;
    // measured: one per W load costs ~25% of the streaming rate); shorter on
    // ties.  GW = 5 serves vocabularies just over 4 x 128 rows per CU (V =
    // 152064: 238 tiles of 640 rows in one round instead of 4-5 tiles of 128).
    const int cus = std::min(device_cu_count(), MAX_WG);
    int best_gw = 4;
    double best = 1e30;
    for (int gw : {4, 5, 2, 1}) {
      const long tiles = (a.V + 128L * gw - 1) / (128L * gw);
      const double t = (double)((tiles + cus - 1) / cus) * gw * (1.0 + 0.25 / gw);
      if (t < best - 1e-9) {
        best = t;
        best_gw = gw;
      }
    }
    const int grid = (int)std::min<long>((a.V + 128L * best_gw - 1) / (128L * best_gw), cus);
    if (best_gw == 5)
      hipLaunchKernelGGL((head_stream_kernel<5, 8>), dim3(grid), dim3(256), 0, s, a);
    else if (best_gw == 4)
      hipLaunchKernelGGL((head_stream_kernel<4, 8>), dim3(grid), dim3(256), 0, s, a);
    else if (best_gw == 2)
      hipLaunchKernelGGL((head_stream_kernel<2, 16>), dim3(grid), dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL((head_stream_kernel<1, 16>), dim3(grid), dim3(256), 0, s, a);
  } else if (rg > 2) {
    // register-direct vocabulary rows (65..256 head rows): 256-row vocabulary
    // tiles spread evenly over at most one workgroup per CU
    const int ntiles = (a.V + HEAD_TILE - 1) / HEAD_TILE, cus = std::min(device_cu_count(), MAX_WG);
    const int per = (ntiles + cus - 1) / cus, grid = (ntiles + per - 1) / per;
    // the variant that also stores the logits (a debug buffer) is its own kernel
    auto go1 = [&](auto tic, auto lgc) {
      constexpr int TI = decltype(tic)::value;
      constexpr bool LG = decltype(lgc)::value;
      constexpr size_t lds = (size_t)4 * TI * 32 * 128;
      static const hipError_t attr = hipFuncSetAttribute((const void*)head_wd_kernel<TI, LG>,
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      hip_check(attr, "hipFuncSetAttribute(head_wd)");
      hipLaunchKernelGGL((head_wd_kernel<TI, LG>), dim3(grid), dim3(256), lds, s, a);
    };
    auto go = [&](auto tic) {
      if (a.logits)
        go1(tic, std::true_type{});
      else
        go1(tic, std::false_type{});
    };
    if (rg <= 4)
      go(std::integral_constant<int, 4>{});
    else
      go(std::integral_constant<int, 8>{});
  } else if (rg <= 1) HeadCfg<1, 256, 8, 4>::launch(a, s);
  else HeadCfg<2, 256, 8, 3>::launch(a, s);
  DLLM_LAUNCH_CHECK("head_bf16");
}

}  // namespace dllm
