// bf16 GEMM on CDNA4 matrix cores with the step's fused epilogues.
//
//   C[M, N] = A[M, K] * Bv[N, K]^T       (both operands K-contiguous, fp32 accumulate)
//
// Bv is a "virtual" weight matrix whose rows come from up to three tensors, so
// q/k/v and gate/up never need to be concatenated in memory:
//   QKV    : rows [0, n0) of Wq, then n1 rows of Wk, then Wv; inside each q and k
//            head the rows are reordered so that every 32-row block holds 16
//            dimensions d and the matching d + 64 (the rotate-half pair).  The
//            epilogue applies RoPE and writes q [B,Hq,L,hd], k [B,Hkv,L,hd] as
//            bf16 and v^T [B,Hkv,hd,L] as the bf16-rounded values in IEEE half.
//   SWIGLU : 16-row chunks alternate between Wgate and Wup (gate rows f..f+15,
//            then up rows f..f+15); the epilogue writes silu(gate) * up as bf16
//            [M, F].
//   RESID  : plain W; the epilogue adds the result to the float32 residual.
//
// Tiling: BM x BN x 64 per workgroup of 4 or 8 wavefronts, each wave owning a
// 64 x 128 or 64 x 96 block of 32x32 MFMA tiles (v_mfma_f32_32x32x16_bf16).
// Tiles of A and Bv stream from memory straight into a 2- or 3-stage LDS ring
// (buffer_load_dwordx4 ... lds, no staging registers), with one barrier per
// k-step.  LDS rows are 128 bytes (64 bf16); the 16-byte chunk c of row r is
// stored at slot c ^ ((r >> 1) & 7), so the sixteen rows read by sixteen
// consecutive lanes cover all 64 LDS banks.
//
// MFMA register layouts (64 lanes, lane = l):
//   A operand : row l%32, k = 8*(l/32) .. +7       B operand : col l%32, same k
//   D (16 x f32): col l%32, row 8*(r/4) + 4*(l/32) + r%4 for register r
//
// Split-K (RESID only): grid.z slices of K write float32 partial tiles; a second
// kernel adds them to the residual in slice order (deterministic, no atomics).
#include "kernels.h"

namespace dllm {

namespace {

constexpr int BK = 64;

// Virtual weight row n -> (tensor index, row inside that tensor).  Every 32-row
// block of the virtual matrix is self-contained for its epilogue: its rows 0..15
// and 16..31 are the two operands that meet in one output (gate and up of the
// same 16 columns f; the rotate-half pair d and d + 64 of the same head for q
// and k), so the pair sits in lanes l and l ^ 16 of one MFMA result and any
// wave tile that is a multiple of 32 columns wide can finish it.  Region
// boundaries (Hq*hd, Hkv*hd rows) are multiples of 128, so no 8-row DMA group
// crosses tensors.
template <int EPI>
__device__ __forceinline__ int2 vrow(const GemmArgs& g, int n) {
  if (EPI == EPI_QKV_ROPE) {
    int t = 0;
    if (n >= g.n0 + g.n1) {
      return make_int2(2, n - g.n0 - g.n1);  // v: identity
    } else if (n >= g.n0) {
      t = 1;
      n -= g.n0;
    }
    const int c = n & 127, blk = c >> 5, w = c & 31;
    const int dim = (w < 16) ? 16 * blk + w : 64 + 16 * blk + (w - 16);
    return make_int2(t, (n & ~127) + dim);
  }
  if (EPI == EPI_SWIGLU) {
    const int chunk = n >> 4;
    return make_int2(chunk & 1, ((chunk >> 1) << 4) + (n & 15));
  }
  return make_int2(0, n);
}

// 16-byte chunk c of 128-byte LDS row r lives in slot c ^ ((r >> 1) & 7): the
// 16 consecutive rows that one 16-lane pass of ds_read_b128 touches then cover
// all 64 banks (two rows per 256-byte bank line, eight slots each).
__device__ __forceinline__ int swz(int row, int chunk) { return row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4); }

// KG = 2 splits every k-step between two groups of waves that own the same
// output blocks (group g takes the k-slices 2g, 2g + 1 of each 64-wide step):
// a tile that four waves would cover then runs two waves per SIMD, so one
// wave's LDS reads overlap the other's MFMAs, at the LDS bytes per flop of the
// four-wave tile.  The second group's accumulators are added to the first's
// through LDS after the main loop.
template <int BM_, int BN_, int WAVES_M, int WAVES_N, int STAGES_, int KG_ = 1>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, S = STAGES_, KG = KG_;
  static constexpr int NWT = WAVES_M * WAVES_N;             // waves per k-group (one output block each)
  static constexpr int NW = NWT * KG, NTH = 64 * NW;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int TI = WM / 32, TJ = WN / 32;          // MFMA tiles per wave
  static constexpr int IA = BM / 8 / NW, IB = BN / 8 / NW;   // LDS-DMA instructions per wave per stage
  static constexpr int LDS_STAGE = (BM + BN) * 128;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tiles are whole 32 x 32 MFMA blocks");
  static_assert(IA * NW * 8 == BM && IB * NW * 8 == BN, "tile rows must split evenly over the DMA loads");
  static_assert(NW % 2 == 0, "the DMA swizzle assumes an even wave count");
  static_assert(KG == 1 || KG == 2, "one or two k-groups");
};
// 128 x 256, 4 waves of 64 x 128, three stages (small M: more tiles to spread over 256 CUs)
using TileS = Tile<128, 256, 2, 2, 3>;
// 256 x 256, 8 waves of 64 x 128 (two per SIMD), two stages (large M: fewer bytes per flop)
using TileL = Tile<256, 256, 4, 2, 2>;
// 256 x 192, 8 waves of 64 x 96: at M = 512, N = 24576 it makes exactly 256 tiles
using TileM = Tile<256, 192, 4, 2, 2>;
// 128 x 192, 4 waves of 64 x 96, three stages
using TileSM = Tile<128, 192, 2, 2, 3>;
// the same on 8 waves in two k-groups
using TileSM2 = Tile<128, 192, 2, 2, 3, 2>;
// 128 x 128, 8 waves of 64 x 64 in two k-groups, four stages
using TileQ = Tile<128, 128, 2, 2, 4, 2>;
// 64 x 256, 8 waves of 64 x 64 in two k-groups: launches of a
// few dozen rows (a cached step's block rows), where the weights' HBM stream
// bounds the time and taller tiles only add MFMA and LDS work on padding rows
using TileT = Tile<64, 256, 1, 4, 4, 2>;  // four stages: three k-steps of weights in flight

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Wait until at most N of this wave's vector-memory operations are in flight
// (gfx9 s_waitcnt encoding: vmcnt split over bits 3:0 and 15:14, expcnt and
// lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// The same with lgkmcnt(0): this wave's LDS reads (and writes) have completed.
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier without the memory-model fence of __syncthreads (which
// would wait for every in-flight LDS-DMA load); the asm clobbers keep the
// compiler from moving memory operations across it.  Callers wait for their
// own DMA loads with wait_vmcnt first.
__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// XCD-aware, grouped tile order: linear position lin -> tile origin (m0, n0).
// The order walks groups of up to GM M-tiles across all N-tiles, so tiles that
// run together share a few A tiles and a few weight tiles in L2.
template <class TL>
__device__ __forceinline__ int2 tile_origin(const GemmArgs& g, int lin) {
  constexpr int GM = 8;
  const int mt = (g.M + TL::BM - 1) / TL::BM, ntl = g.N / TL::BN;
  const int grp = lin / (GM * ntl), first_m = grp * GM, gsize = min(mt - first_m, GM);
  const int in_grp = lin - grp * GM * ntl;
  return make_int2((first_m + in_grp % gsize) * TL::BM, (in_grp / gsize) * TL::BN);
}

// acc += A[m0 : m0+BM, k] * Bv[n0 : n0+BN, k]^T over the k-steps kt0 .. kt0+nk-1
// (64 wide), streamed through the S-stage LDS ring.  Starts with a barrier, so
// the ring may still be in use by a previous call; leaves no load in flight.
// PB: Bv is read from its packed copy g.Wp (pack_gemm_weights_kernel), where
// the tile's 256 rows x 64 k of a k-step are one contiguous 32 KiB run whose
// 1 KiB pieces are the MFMA B operands of (32-row group, 16-k slice) in lane
// order: the DMA streams whole runs and each fragment read is lane-linear.
template <class TL, int EPI, bool PB = false>
__device__ __forceinline__ void mma_tile(const GemmArgs& g, char* lds, int wave, int lane, int m0, int n0, int kt0,
                                         int nk, f32x16_t (&acc)[TL::TI][TL::TJ]) {
  static_assert(!PB || TL::BN == 256, "a packed tile is one 256-row tile of the copy");
  constexpr int BM = TL::BM, BN = TL::BN, S = TL::S, NW = TL::NW;
  const int wt = wave % TL::NWT, kg = wave / TL::NWT;
  const int wm = wt / (BN / TL::WN), wn = wt % (BN / TL::WN);
  const int kbeg = kt0 * BK;

  // LDS-DMA loads: instruction i of wave w fills tile rows 8 (NW i + w) .. +7
  // (1 KiB of LDS).  Lane l writes row + l/8, slot l%8, which holds the row's
  // logical 16-byte chunk (l%8) ^ ((row >> 1) & 7); with NW even, row >> 1
  // = 4 (w & 1) + (l/8) / 2 modulo 8, the same for every i.
  // Row offsets are fixed across k; the k advance goes in the scalar offset.
  // A rows past M are clamped to M-1 (their results are never stored).
  const int lr = lane >> 3, lc = (lane & 7) ^ (((wave & 1) << 2) | (lr >> 1));
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc((void*)g.A, 0, 0x7fffffff, 0x00020000);
  // In 8-wave tiles only waves 0..3 (one per SIMD) issue the DMA, each for its
  // own rows and those of wave + 4: an LDS-DMA burst stalls the issuing wave,
  // and the other wave of its SIMD keeps the MFMA pipe busy meanwhile (gate/up
  // at M = 8192: 1496 -> 1415 us; 1-4% at M = 512).  wave + 4 has the same
  // parity, so the same chunk swizzle.
  constexpr int HW = NW == 8 ? 2 : 1;  // waves whose DMA one issuing wave covers
  const bool issuer = HW == 1 || wave < NW / 2;
  uint32_t voa[HW][TL::IA];
#pragma unroll
  for (int hw = 0; hw < HW; ++hw)
#pragma unroll
    for (int i = 0; i < TL::IA; ++i) {
      const int wv = wave + hw * (NW / 2);
      const int row = min(m0 + 8 * (NW * i + wv) + lr, g.M - 1);
      voa[hw][i] = (uint32_t)(((size_t)row * g.K + kbeg + lc * 8) * 2);
    }
  // Bv rows: each 8-row DMA group lies in one tensor (the tile's q/k/v tensor,
  // or gate / up by 32-row parity for SwiGLU).
  const bf16_t* wsrc[3] = {g.W0, g.W1, g.W2};
  __amdgpu_buffer_rsrc_t rbs[HW][TL::IB];
  uint32_t vob[HW][TL::IB];
#pragma unroll
  for (int hw = 0; hw < HW; ++hw)
#pragma unroll
    for (int i = 0; i < TL::IB; ++i) {
      const int wv = wave + hw * (NW / 2);
      if (PB) {
        // piece NW i + w of the (n0 / 256, k-step) run; the k advance is 32 KiB per step
        rbs[hw][i] = __builtin_amdgcn_make_buffer_rsrc((void*)g.Wp, 0, 0x7fffffff, 0x00020000);
        vob[hw][i] = (uint32_t)((((size_t)(n0 >> 8) * (g.K / BK) + kt0) * 32768) + (NW * i + wv) * 1024 + lane * 16);
      } else {
        const int2 first = vrow<EPI>(g, n0 + 8 * (NW * i + wv));  // wave-uniform
        rbs[hw][i] = __builtin_amdgcn_make_buffer_rsrc((void*)wsrc[first.x], 0, 0x7fffffff, 0x00020000);
        vob[hw][i] = (uint32_t)(((size_t)(first.y + lr) * g.K + kbeg + lc * 8) * 2);
      }
    }
  auto issue = [&](int kt) {
    if (!issuer) return;
    char* base = lds + (kt % S) * TL::LDS_STAGE;
    const int soff = kt * BK * 2, soff_b = PB ? kt * 32768 : soff;
#pragma unroll
    for (int hw = 0; hw < HW; ++hw) {
      const int wv = wave + hw * (NW / 2);
#pragma unroll
      for (int i = 0; i < TL::IA; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(base + 8 * (NW * i + wv) * 128), 16, voa[hw][i],
                                                 soff, 0, 0);
#pragma unroll
      for (int i = 0; i < TL::IB; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rbs[hw][i], (lds_ptr_t)(base + BM * 128 + 8 * (NW * i + wv) * 128),
                                                 16, vob[hw][i], soff_b, 0, 0);
    }
  };

  constexpr int PER_STAGE = HW * (TL::IA + TL::IB);  // DMA instructions per issuing wave per stage
  constexpr int NS = BK / 16, NF = TL::TI + TL::TJ, NM = TL::TI * TL::TJ;
  constexpr int NSW = NS / TL::KG;  // k-slices of a step that this wave's group computes
  static_assert(NM >= NF && NSW % 2 == 0, "pipeline needs at least as many MFMAs as fragment reads per slice");
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int ks0 = kg * NSW;  // the group's first slice (even, so register sets alternate across steps)

  // Fragments of the group's 16-wide k-slices of a tile go through two
  // register sets: slice kl + 1 is read while the MFMAs of slice kl run.  The
  // barrier that publishes tile kt + 1 sits before the group's last slice of
  // tile kt, so the first fragments of tile kt + 1 are read under that slice's
  // MFMAs and the k-step boundary costs no exposed LDS latency; the slot tile
  // kt occupied is refilled (tile kt + S) right after that barrier.
  bf16x8_t af[2][TL::TI], bfr[2][TL::TJ];
  auto frag = [&](const char* base, int kl) {
    const int ch = (ks0 + kl) * 2 + lhalf, set = kl & 1;
#pragma unroll
    for (int i = 0; i < TL::TI; ++i)
      af[set][i] = *reinterpret_cast<const bf16x8_t*>(base + swz(wm * TL::WM + i * 32 + lrow, ch));
#pragma unroll
    for (int j = 0; j < TL::TJ; ++j)
      bfr[set][j] = PB ? *reinterpret_cast<const bf16x8_t*>(
                             base + BM * 128 + ((((wn * TL::WN + j * 32) >> 5) * 4 + ks0 + kl) << 10) + lane * 16)
                       : *reinterpret_cast<const bf16x8_t*>(base + BM * 128 + swz(wn * TL::WN + j * 32 + lrow, ch));
  };

  wait_vm_lds<0>();
  barrier_nofence();  // every wave is done with the ring's previous contents
#pragma unroll
  for (int s = 0; s < S; ++s)
    if (s < nk) issue(s);
  // this wave's loads of tile 0 are done once only the later tiles' are outstanding
  if (nk >= S)
    wait_vm_lds<PER_STAGE * (S - 1)>();
  else
    wait_vm_lds<0>();
  barrier_nofence();
  frag(lds, 0);

  for (int kt = 0; kt < nk; ++kt) {
    const char* base = lds + (kt % S) * TL::LDS_STAGE;
#pragma unroll
    for (int ks = 0; ks < NSW; ++ks) {
      bool next = false;
      if (ks + 1 < NSW) {
        frag(base, ks + 1);
        next = true;
      } else if (kt + 1 < nk) {
        // tile kt + 1 has landed once only tiles kt + 2 .. kt + S - 1 are
        // outstanding; every LDS read of tile kt has completed (lgkmcnt 0)
        if (kt + S - 1 < nk)
          wait_vm_lds<PER_STAGE * (S - 2)>();
        else
          wait_vm_lds<0>();
        barrier_nofence();  // tile kt + 1 visible to all waves; slot kt % S free
        if (kt + S < nk) issue(kt + S);
        frag(lds + ((kt + 1) % S) * TL::LDS_STAGE, 0);
        next = true;
      }
#pragma unroll
      for (int i = 0; i < TL::TI; ++i)
#pragma unroll
        for (int j = 0; j < TL::TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks & 1][i], bfr[ks & 1][j], acc[i][j], 0, 0, 0);
      if (next) {
#pragma unroll
        for (int x = 0; x < NF; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA of slice ks
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one fragment read of the next slice
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM - NF, 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
      }
    }
  }
}

// Epilogue of one unit of a tile for the float32 residual (or a plain bf16
// store): the accumulator rows 8c .. 8c+7 ... that a lane holds for row block
// i, i.e. v[j][e] = acc[i][j][4c + e] for the TJ column blocks j of the wave
// (rows 8c + 4 (lane/32) + e, columns j*32 + lane%32 of the wave's 32-row
// block i); 32 lanes cover 128 contiguous bytes of a residual row.
template <class TL, int EPI>
__device__ __forceinline__ void epi_unit(const GemmArgs& g, int wave, int lane, int m0, int n0, int i, int c,
                                         const float (&v)[TL::TJ][4]) {
  const int wm = (wave % TL::NWT) / (TL::BN / TL::WN), wn = (wave % TL::NWT) % (TL::BN / TL::WN);
  const int lhalf = lane >> 5, col_in = lane & 31;
  const int mrow = m0 + wm * TL::WM + i * 32 + 8 * c + 4 * lhalf;  // + e
  const int ncol0 = n0 + wn * TL::WN;                               // + j*32 + col_in
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int m = mrow + e;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < TL::TJ; ++j) {
      const int n = ncol0 + j * 32 + col_in;
      if (EPI == EPI_RESID)
        g.resid[(size_t)m * g.N + n] += v[j][e];
      else
        g.out[(size_t)m * g.N + n] = f2bf(v[j][e]);
    }
  }
}

// LDS staging of the SwiGLU and q/k/v epilogues.  Their outputs are 16-bit and,
// written straight from the MFMA layout, would go out as 2-byte stores (v^T
// even touching 32 cache lines per instruction).  Instead each wave writes its
// finished values into the LDS ring (free once the main loop is done) in the
// destination's order, and the workgroup then stores 16-byte chunks.
template <int BM, int BN>
struct StageGeo {
  // SwiGLU: [BM][BN/2] bf16, rows padded by 16 bytes (conflict-free writes)
  static constexpr int SW_ROW = BN + 16;
  static constexpr int SW_BYTES = BM * SW_ROW;
  // q/k/v: one area per 32-column block; a q/k block holds [BM][32] bf16
  // (64-byte rows: dimensions d .. d+15, then d+64 .. d+79), a v block
  // [32][BM] half (v^T, each column padded by 16 bytes)
  static constexpr int VROW = (BM + 8) * 2;
  static constexpr int BLK = (BM * 64 > 32 * VROW) ? BM * 64 : 32 * VROW;
  static constexpr int QKV_BYTES = BN / 32 * BLK;
};
template <class TL>
struct Stage : StageGeo<TL::BM, TL::BN> {};

// k-group merge area: the second group's accumulators, [NWT][TI*TJ][4][64 lanes] float4
template <class TL>
constexpr size_t merge_bytes() {
  return TL::KG == 1 ? 0 : (size_t)TL::NWT * TL::TI * TL::TJ * 4 * 64 * 16;
}

template <class TL, int EPI>
constexpr size_t lds_bytes() {
  const size_t ring = (size_t)TL::S * TL::LDS_STAGE;
  const size_t st = EPI == EPI_SWIGLU ? Stage<TL>::SW_BYTES : EPI == EPI_QKV_ROPE ? Stage<TL>::QKV_BYTES : 0;
  const size_t mg = merge_bytes<TL>();
  const size_t a = ring > st ? ring : st;
  return a > mg ? a : mg;
}

// The value lane l ^ 16 holds (v_permlane16_swap: a VALU exchange of the odd
// and even 16-lane rows; with both operands equal its two results are the
// values of the lower and the upper row at this position).
__device__ __forceinline__ float swap16(float x, bool hi) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(hi ? r[0] : r[1]);
}

// v is stored for the attention kernel's half-precision P.V product as the IEEE
// half of its bf16 value: exact for 2^-17 <= |v| <= 65504 (bf16's 8-bit
// significand fits half's; below, half's subnormal step 2^-24 bounds the
// error).  A bf16 value beyond 65504 (i.e. >= 65536) is stored as +-65504 and
// flagged in the error word.
__device__ __forceinline__ f16_t v_half(float x, bool& over) {
  const float b = bf2f(f2bf(x));
  if (fabsf(b) > 65504.f) {
    over = true;
    return f2h(copysignf(65504.f, b));
  }
  return f2h(b);
}

// (sequence, position) of token row m = b L + pos, by a float reciprocal and a
// one-step fixup: exact for m < 2^24 and B < 2^16 (the estimate of m / L is
// then off by less than one), several times cheaper than an integer division.
__device__ __forceinline__ int2 seq_pos(int m, int L, float inv_l) {
  int b = (int)((float)m * inv_l);
  int p = m - b * L;
  if (p < 0) {
    p += L;
    --b;
  } else if (p >= L) {
    p -= L;
    ++b;
  }
  return make_int2(b, p);
}

// Store phase of the staged epilogues: the workgroup's NTH threads write the
// staged tile (StageGeo layout) to its destination as 16-byte chunks.
template <int BM, int BN, int NTH, int EPI>
__device__ __forceinline__ void staged_store(const GemmArgs& g, const char* lds, int m0, int n0) {
  using St = StageGeo<BM, BN>;
  constexpr int HD = 128, HALF = 64;
  const int nq = g.Hq * HD, nkv = g.Hkv * HD;
  const float inv_l = 1.0f / (float)g.Lq;  // rows per sequence
  const int tid = threadIdx.x;
  if (EPI == EPI_SWIGLU) {
    const int F = g.N / 2, f0 = n0 / 2;
    constexpr int CH = BN / 16;  // 16-byte chunks per row
    for (int it = tid; it < BM * CH; it += NTH) {
      const int r = it / CH, q = it - r * CH, m = m0 + r;
      if (m < g.M)
        *reinterpret_cast<uint4*>(g.out + (size_t)m * F + f0 + 8 * q) =
            *reinterpret_cast<const uint4*>(lds + r * St::SW_ROW + 16 * q);
    }
    return;
  }
#pragma unroll 1
  for (int jb = 0; jb < BN / 32; ++jb) {
    const int vb = n0 + jb * 32;
    const char* blk = lds + jb * St::BLK;
    if (vb < nq + nkv) {
      const bool isq = vb < nq;
      const int rel = isq ? vb : vb - nq;
      const int head = rel / HD, d0 = 16 * ((rel % HD) >> 5);
      // q [B, Hq, Lq, hd] at row i; k [B, Hkv, L, hd] at position pos0 + i
      const int H = isq ? g.Hq : g.Hkv, LL = isq ? g.Lq : g.L, p0 = isq ? 0 : g.pos0;
      bf16_t* dst = isq ? g.q : g.k;
      for (int it = tid; it < BM * 4; it += NTH) {
        const int r = it >> 2, q = it & 3, m = m0 + r;
        if (m >= g.M) continue;
        const int2 bp = seq_pos(m, g.Lq, inv_l);
        const int b = bp.x, pos = p0 + bp.y;
        const int dim = (q < 2 ? d0 : HALF + d0) + 8 * (q & 1);
        *reinterpret_cast<uint4*>(dst + (((size_t)b * H + head) * LL + pos) * HD + dim) =
            *reinterpret_cast<const uint4*>(blk + r * 64 + 16 * q);
      }
    } else {
      const int rel = vb - nq - nkv;
      const int head = rel / HD, cj0 = rel % HD;
      constexpr int RC = BM / 8;  // 8-row chunks per column
      for (int it = tid; it < 32 * RC; it += NTH) {
        const int c = it / RC, t = it - c * RC, m = m0 + 8 * t;
        if (m >= g.M) continue;
        const uint4 val = *reinterpret_cast<const uint4*>(blk + c * St::VROW + 16 * t);
        if (((g.L | g.Lq | g.pos0) & 7) == 0 && m + 7 < g.M) {
          // eight positions of one sequence, 16-byte aligned (L, Lq, pos0 and m
          // multiples of 8)
          const int2 bp = seq_pos(m, g.Lq, inv_l);
          const int b = bp.x, pos = g.pos0 + bp.y;
          *reinterpret_cast<uint4*>(g.vt + (((size_t)b * g.Hkv + head) * HD + cj0 + c) * g.L + pos) = val;
        } else {
          const uint32_t wd[4] = {val.x, val.y, val.z, val.w};
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int mm = m + e;
            if (mm >= g.M) break;
            const int2 bp = seq_pos(mm, g.Lq, inv_l);
            const int b = bp.x, pos = g.pos0 + bp.y;
            g.vt[(((size_t)b * g.Hkv + head) * HD + cj0 + c) * g.L + pos] = (f16_t)(wd[e >> 1] >> (16 * (e & 1)));
          }
        }
      }
    }
  }
}

template <class TL, int EPI>
__device__ __forceinline__ void epilogue_staged(const GemmArgs& g, char* lds, int wave, int lane, int m0, int n0,
                                                const f32x16_t (&acc)[TL::TI][TL::TJ]) {
  using St = Stage<TL>;
  constexpr int HD = 128, HALF = 64;
  const int wm = (wave % TL::NWT) / (TL::BN / TL::WN), wn = (wave % TL::NWT) % (TL::BN / TL::WN);
  const int lhalf = lane >> 5, col_in = lane & 31, w = col_in & 15;
  // For SwiGLU and q/k the two operands of an output sit in lanes l and l ^ 16
  // (see vrow): after one exchange of two values the lane with column < 16
  // holds both operands of rows e = 0, 1 and its partner those of rows 2, 3.
  const bool hi = col_in >= 16;
  const int e0 = hi ? 2 : 0;
  const int nq = g.Hq * HD, nkv = g.Hkv * HD;

  wait_vm_lds<0>();
  barrier_nofence();  // every wave is done reading the ring

  const float inv_l = 1.0f / (float)g.Lq;  // rows per sequence
  bool v_over = false;
  // with two k-groups only the first holds the finished tile; the second
  // joins the barriers and the stores
  if (wave < TL::NWT) {
#pragma unroll
  for (int i = 0; i < TL::TI; ++i) {
    // q/k: the RoPE table values of this lane's two finished rows in each of
    // the four 8-row groups of row block i, for every q/k column block, all
    // loaded before the first is used
    float cs[4][TL::TJ][2], sn[4][TL::TJ][2];
    if (EPI == EPI_QKV_ROPE) {
      int pos[4][2];
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          // rows past M are staged but never stored
          const int m = min(m0 + wm * TL::WM + i * 32 + 8 * c + 4 * lhalf + e0 + k, g.M - 1);
          pos[c][k] = g.pos0 + seq_pos(m, g.Lq, inv_l).y;
        }
#pragma unroll
      for (int j = 0; j < TL::TJ; ++j) {
        const int vb = n0 + wn * TL::WN + j * 32;
        if (vb >= nq + nkv) continue;
        const int rel = vb < nq ? vb : vb - nq;
        const int d = 16 * ((rel % HD) >> 5) + w;
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            cs[c][j][k] = g.cosb[(size_t)pos[c][k] * HALF + d];
            sn[c][j][k] = g.sinb[(size_t)pos[c][k] * HALF + d];
          }
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int rl0 = wm * TL::WM + i * 32 + 8 * c + 4 * lhalf;  // tile row of e = 0
#pragma unroll
      for (int j = 0; j < TL::TJ; ++j) {
        const int tcol = wn * TL::WN + j * 32;  // tile column of the block (wave-uniform)
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * c + e];
        const bool pair = EPI == EPI_SWIGLU || n0 + tcol < nq + nkv;
        float own[2] = {0.f, 0.f}, oth[2] = {0.f, 0.f};
        if (pair) {
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const float send = hi ? v[k] : v[2 + k];  // the rows the partner finishes
            own[k] = hi ? v[2 + k] : v[k];
            oth[k] = swap16(send, hi);
          }
        }
        if (EPI == EPI_SWIGLU) {  // lo lanes hold gate, hi lanes up
          const int fl = (tcol >> 1) + w;
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const float gt = hi ? oth[k] : own[k], up = hi ? own[k] : oth[k];
            // silu with the hardware exp2 and reciprocal: the result is rounded to bf16
            *reinterpret_cast<bf16_t*>(lds + (rl0 + e0 + k) * St::SW_ROW + fl * 2) =
                f2bf(__fdividef(gt, 1.0f + __expf(-gt)) * up);
          }
        } else {
          char* blk = lds + (tcol >> 5) * St::BLK;
          if (pair) {  // q or k: lo lanes hold x1 = dimension d, hi lanes x2 = d + 64
#pragma unroll
            for (int k = 0; k < 2; ++k) {
              const int rl = rl0 + e0 + k;
              const float x1 = hi ? oth[k] : own[k], x2 = hi ? own[k] : oth[k];
              const float c_ = cs[c][j][k], s_ = sn[c][j][k];
              *reinterpret_cast<bf16_t*>(blk + rl * 64 + w * 2) = f2bf(x1 * c_ - x2 * s_);
              *reinterpret_cast<bf16_t*>(blk + rl * 64 + (16 + w) * 2) = f2bf(x2 * c_ + x1 * s_);
            }
          } else {  // v: four consecutive rows of column col_in, as IEEE half of the bf16 value
            uint2 pk;
            pk.x = (uint32_t)v_half(v[0], v_over) | ((uint32_t)v_half(v[1], v_over) << 16);
            pk.y = (uint32_t)v_half(v[2], v_over) | ((uint32_t)v_half(v[3], v_over) << 16);
            *reinterpret_cast<uint2*>(blk + col_in * St::VROW + rl0 * 2) = pk;
          }
        }
      }
    }
  }

  }
  if (EPI == EPI_QKV_ROPE && v_over && g.err) atomicOr(g.err, (int)ERR_V_RANGE);

  __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
  barrier_nofence();

  staged_store<TL::BM, TL::BN, TL::NTH, EPI>(g, lds, m0, n0);
}

// Writes the finished tile at (m0, n0) from the accumulators.
template <class TL, int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& g, int wave, int lane, int m0, int n0,
                                         const f32x16_t (&acc)[TL::TI][TL::TJ]) {
#pragma unroll
  for (int i = 0; i < TL::TI; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float v[TL::TJ][4];
#pragma unroll
      for (int j = 0; j < TL::TJ; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[j][e] = acc[i][j][4 * c + e];
      epi_unit<TL, EPI>(g, wave, lane, m0, n0, i, c, v);
    }
}

template <class TL>
__device__ __forceinline__ void zero_acc(f32x16_t (&acc)[TL::TI][TL::TJ]) {
#pragma unroll
  for (int i = 0; i < TL::TI; ++i)
#pragma unroll
    for (int j = 0; j < TL::TJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
}

// One workgroup per output tile (grid.x), optionally split over K (grid.z:
// float32 partial tiles, summed by splitk_resid_kernel).
template <class TL, int EPI, bool PB = false>
__global__ void __launch_bounds__(TL::NTH, 1) gemm_bf16_kernel(GemmArgs g) {
  // The buffer-resource builtins exist only for the device target; the host
  // pass needs just the kernel's signature for its launch stub.
#if defined(__HIP_DEVICE_COMPILE__)
  extern __shared__ __attribute__((aligned(16))) char lds[];
  // wave index made provably uniform so per-wave buffer descriptors stay scalar
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tiles = ((g.M + TL::BM - 1) / TL::BM) * (g.N / TL::BN);
  // workgroup i (in x, then z order) runs on XCD i % 8: give each XCD a
  // contiguous run of the (split, tile) order -- XCD x takes T / 8 of the
  // T = tiles x splits workgroups, one more for the first T % 8 XCDs
  const int T = tiles * (int)gridDim.z, i = blockIdx.x + tiles * blockIdx.z, x = i & 7;
  const int li = x * (T >> 3) + min(x, T & 7) + (i >> 3);
  const int lin = li % tiles, zs = li / tiles;
  const int2 o = tile_origin<TL>(g, lin);
  // K slice z of S: k-steps [z KS / S, (z + 1) KS / S)
  const int ks_total = g.K / BK;
  const int kt0 = (int)((long)zs * ks_total / gridDim.z);
  const int nk = (int)((long)(zs + 1) * ks_total / gridDim.z) - kt0;

  f32x16_t acc[TL::TI][TL::TJ];
  zero_acc<TL>(acc);
  mma_tile<TL, EPI, PB>(g, lds, wave, lane, o.x, o.y, kt0, nk, acc);

  if (TL::KG == 2) {
    // acc(group 0) += acc(group 1) through LDS (the ring is idle once every
    // wave has passed the barrier); lane-contiguous float4 rows
    wait_vm_lds<0>();
    barrier_nofence();
    float4* xa = reinterpret_cast<float4*>(lds) + (size_t)(wave % TL::NWT) * (TL::TI * TL::TJ * 4 * 64) + lane;
    if (wave >= TL::NWT) {
#pragma unroll
      for (int i = 0; i < TL::TI; ++i)
#pragma unroll
        for (int j = 0; j < TL::TJ; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            xa[((i * TL::TJ + j) * 4 + q) * 64] =
                make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
    }
    wait_vm_lds<0>();
    barrier_nofence();
    if (wave < TL::NWT) {
#pragma unroll
      for (int i = 0; i < TL::TI; ++i)
#pragma unroll
        for (int j = 0; j < TL::TJ; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float4 v = xa[((i * TL::TJ + j) * 4 + q) * 64];
            acc[i][j][4 * q] += v.x;
            acc[i][j][4 * q + 1] += v.y;
            acc[i][j][4 * q + 2] += v.z;
            acc[i][j][4 * q + 3] += v.w;
          }
    }
    // the staged epilogues have barriers: every wave takes part; the others
    // are done
    if (wave >= TL::NWT && !(gridDim.z == 1 && (EPI == EPI_SWIGLU || EPI == EPI_QKV_ROPE))) return;
  }

  if (gridDim.z > 1) {  // split-K partial tile
    const int wm = (wave % TL::NWT) / (TL::BN / TL::WN), wn = (wave % TL::NWT) % (TL::BN / TL::WN);
    const int lhalf = lane >> 5, col_in = lane & 31;
    float* part = g.splitk_buf + (size_t)zs * g.M * g.N;
#pragma unroll
    for (int i = 0; i < TL::TI; ++i)
#pragma unroll
      for (int j = 0; j < TL::TJ; ++j) {
        const int n = o.y + wn * TL::WN + j * 32 + col_in;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = o.x + wm * TL::WM + i * 32 + 8 * (r >> 2) + 4 * lhalf + (r & 3);
          if (m < g.M) part[(size_t)m * g.N + n] = acc[i][j][r];
        }
      }
    return;
  }
  if (EPI == EPI_SWIGLU || EPI == EPI_QKV_ROPE)
    epilogue_staged<TL, EPI>(g, lds, wave, lane, o.x, o.y, acc);
  else
    epilogue<TL, EPI>(g, wave, lane, o.x, o.y, acc);
#endif
}

// resid[m, n] += sum_z part[z, m, n], z in order.
template <int S>
__global__ void splitk_resid_kernel(const float* __restrict__ part, float* __restrict__ resid, long MN) {
  const long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= MN) return;
  float4 acc = *reinterpret_cast<const float4*>(part + i);
#pragma unroll
  for (int z = 1; z < S; ++z) {
    const float4 v = *reinterpret_cast<const float4*>(part + (size_t)z * MN + i);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  float4 h = *reinterpret_cast<float4*>(resid + i);
  h.x += acc.x; h.y += acc.y; h.z += acc.z; h.w += acc.w;
  *reinterpret_cast<float4*>(resid + i) = h;
}

// Split-K epilogues of the SwiGLU and q/k/v GEMMs (launches with few rows):
// the float32 partial tiles [S, M, N] are summed in slice order, then the fused
// epilogues' arithmetic is applied.  One thread per output (SwiGLU) or per
// q/k rotate-half pair / v element.
__global__ void splitk_swiglu_kernel(const float* __restrict__ part, int S, int M, int F,
                                     bf16_t* __restrict__ out) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)M * F) return;
  const int m = (int)(i / F), f = (int)(i - (long)m * F);
  const long N = 2L * F, MN = (long)M * N;
  const long n = (long)m * N + 32 * (f >> 4) + (f & 15);  // gate column; up = n + 16
  float gt = part[n], up = part[n + 16];
  for (int z = 1; z < S; ++z) {
    gt += part[z * MN + n];
    up += part[z * MN + n + 16];
  }
  out[(size_t)m * F + f] = f2bf(__fdividef(gt, 1.0f + __expf(-gt)) * up);
}

__global__ void splitk_qkv_kernel(const float* __restrict__ part, int S, GemmArgs g) {
  constexpr int HD = 128, HALF = 64;
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)g.M * g.N) return;
  const int m = (int)(i / g.N), n = (int)(i - (long)m * g.N);
  const int nq = g.Hq * HD, nkv = g.Hkv * HD;
  const long MN = (long)g.M * g.N;
  const int b = m / g.Lq, r = m - b * g.Lq, pos = g.pos0 + r;
  auto sum = [&](int col) {
    float a = part[(long)m * g.N + col];
    for (int z = 1; z < S; ++z) a += part[z * MN + (long)m * g.N + col];
    return a;
  };
  if (n < nq + nkv) {
    // virtual column n (lower half of its 32-column block) holds dimension d,
    // column n + 16 dimension d + 64 of the same head
    const int w = n & 31;
    if (w >= 16) return;
    const bool isq = n < nq;
    const int rel = isq ? n : n - nq, head = rel / HD, d = 16 * ((rel % HD) >> 5) + w;
    const float x1 = sum(n), x2 = sum(n + 16);
    const float c_ = g.cosb[(size_t)pos * HALF + d], s_ = g.sinb[(size_t)pos * HALF + d];
    bf16_t* dst = isq ? g.q + (((size_t)b * g.Hq + head) * g.Lq + r) * HD : g.k + (((size_t)b * g.Hkv + head) * g.L + pos) * HD;
    dst[d] = f2bf(x1 * c_ - x2 * s_);
    dst[d + HALF] = f2bf(x2 * c_ + x1 * s_);
  } else {
    const int rel = n - nq - nkv, head = rel / HD, cj = rel % HD;
    bool over = false;
    g.vt[(((size_t)b * g.Hkv + head) * HD + cj) * g.L + pos] = v_half(sum(n), over);
    if (over && g.err) atomicOr(g.err, (int)ERR_V_RANGE);
  }
}

// Packed copy of a GEMM's virtual weight matrix Bv [N, K] (rows in vrow order):
// for 256-row tile t and 64-k step kb the block [256, 64] is one contiguous 32
// KiB run, inside it the 1 KiB MFMA operand of 32-row group gr and 16-k slice
// s in lane order (lane l: row 32 gr + l % 32, k 16 s + 8 (l / 32) .. +7) --
// the layout of the LM head's copy.  Rows past N are zero.  One thread per
// 16-byte vector, in destination order.
template <int EPI>
__global__ void pack_gemm_weights_kernel(GemmArgs g, bf16_t* __restrict__ out, size_t nvec) {
  const int nk = g.K / 64;
  const bf16_t* wsrc[3] = {g.W0, g.W1, g.W2};
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < nvec; idx += (size_t)gridDim.x * blockDim.x) {
    const int l = (int)(idx % 64);
    size_t t = idx / 64;
    const int sl = (int)(t % 4);
    t /= 4;
    const int gr = (int)(t % 8);
    t /= 8;
    const int kb = (int)(t % nk);
    const size_t lt = t / nk;
    const int n = (int)(lt * 256 + gr * 32 + (l & 31));
    const int k = kb * 64 + sl * 16 + (l >> 5) * 8;
    bf16x8_t v = {};
    if (n < g.N) {
      const int2 src = vrow<EPI>(g, n);
      v = *reinterpret_cast<const bf16x8_t*>(wsrc[src.x] + (size_t)src.y * g.K + k);
    }
    *reinterpret_cast<bf16x8_t*>(out + idx * 8) = v;
  }
}

// GEMM of at most 64 rows from the packed copy, register-direct (the LM head's
// streaming design): wave w of the grid owns GW 32-row groups of Bv (group
// block w % ngb) and the k-slices [z KS / S, (z + 1) KS / S) of split z =
// w / ngb; per 16-k slice it loads its GW 1 KiB W operands (contiguous runs of
// the copy, non-temporal) and MB X operands (rows 32 mb + l % 32 of A, zero
// past M) into a P-deep register ring -- no LDS, no barrier -- and runs GW x MB
// MFMAs with W as the A operand (a lane ends with 16 columns n of one row m).
// It writes float32 partials part[z, m, n]; the split-K epilogues finish them.
// Loads complete in issue order, so before slice u only the (GW + MB) (P - 1)
// loads of the slices after it may be outstanding.
struct RowsArgs {
  const bf16_t* A;   // [M, K]
  const bf16_t* Wp;  // packed Bv
  float* part;       // [S, M, N]
  int M, N, K, S, ngb;
};

template <int GW, int MB, int P>
__global__ void __launch_bounds__(256, 2) gemm_rows_kernel(RowsArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  static_assert((GW + MB) * (P - 1) < 64, "vmcnt range");
  const int lane = threadIdx.x & 63;
  const int wg = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (wg >= a.ngb * a.S) return;
  const int gb = wg % a.ngb, z = wg / a.ngb;
  const int KS = a.K / 16, nk = a.K / 64;
  const int u0 = (int)((long)z * KS / a.S), n = (int)((long)(z + 1) * KS / a.S) - u0;
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc((void*)a.Wp, 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc((void*)a.A, 0, 0x7fffffff, 0x00020000);
  const int lr = lane & 31, half = lane >> 5;
  // group G = gb GW + j lies in 256-row tile G / 8 at position G % 8
  uint32_t wbase[GW];
#pragma unroll
  for (int j = 0; j < GW; ++j) {
    const int G = gb * GW + j;
    wbase[j] = (uint32_t)(((size_t)(G >> 3) * nk * 8 + (G & 7)) * 4 * 1024 + lane * 16);
  }
  uint32_t xoff[MB];
  bool xok[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = 32 * mb + lr;
    xok[mb] = m < a.M;
    xoff[mb] = (uint32_t)(((size_t)min(m, a.M - 1) * a.K + half * 8) * 2);
  }
  typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
  u32x4_t wbuf[P][GW], xbuf[P][MB];
  auto load = [&](int u, int slot) {
    const int us = u0 + u, kb = us >> 2, sl = us & 3;
#pragma unroll
    for (int j = 0; j < GW; ++j)
      wbuf[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(rw, wbase[j] + (uint32_t)(kb * 32768 + sl * 1024), 0, 2);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      xbuf[slot][mb] = __builtin_amdgcn_raw_buffer_load_b128(rx, xoff[mb] + (uint32_t)(us * 32), 0, 0);
  };
  f32x16_t acc[GW][MB];
#pragma unroll
  for (int j = 0; j < GW; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][mb][r] = 0.f;
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (p < n) load(p, p);
  for (int b0 = 0; b0 < n; b0 += P) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int u = b0 + p;
      if (u < n) {
        if (u + P - 1 < n)
          __builtin_amdgcn_s_waitcnt((((GW + MB) * (P - 1)) & 15) | (7 << 4) | (15 << 8) |
                                     ((((GW + MB) * (P - 1)) >> 4) << 14));
        else
          __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8));  // the last slices: fewer later loads issued
        bf16x8_t xf[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          xf[mb] = __builtin_bit_cast(bf16x8_t, xbuf[p][mb]);
          if (!xok[mb]) xf[mb] = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
        }
#pragma unroll
        for (int j = 0; j < GW; ++j)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
            acc[j][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wbuf[p][j]), xf[mb],
                                                                acc[j][mb], 0, 0, 0);
        if (u + P < n) load(u + P, p);
      }
    }
  }
  // partials: lane holds columns n = 32 G + 8 (r / 4) + 4 half + r % 4 of row m = 32 mb + l % 32
  float* part = a.part + (size_t)z * a.M * a.N;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = 32 * mb + lr;
    if (m >= a.M) continue;
#pragma unroll
    for (int j = 0; j < GW; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int nn = (gb * GW + j) * 32 + 8 * q + 4 * half;
        *reinterpret_cast<float4*>(part + (size_t)m * a.N + nn) =
            make_float4(acc[j][mb][4 * q], acc[j][mb][4 * q + 1], acc[j][mb][4 * q + 2], acc[j][mb][4 * q + 3]);
      }
  }
#endif
}

// Groups per wave and K split of a register-direct launch, by a time model
// measured at 32 rows on the LLaDA-8B shapes: the bytes a compute unit pulls
// bound it (~28 GB/s per CU, 7 per wave), so a launch takes the slices of its
// longest wave x (GW W loads + MB / 4 for the X loads, one costing a quarter
// of a W load) x 0.146 us per KiB, times the workgroups per CU; plus the
// float32 partials written and read back (~8 TB/s).  Fewer splits, then more
// groups per wave, on ties.  Gate/up at 32 rows: 4 groups, split 5 (240
// workgroups: 36 us); with split 6 a second workgroup on 32 of the CUs took 52.
struct RowsPlan {
  int gw, split;
};
RowsPlan rows_plan(int M, int N, int K) {
  const int ng = N / 32, ks = K / 16, mb = M > 32 ? 2 : 1;
  const long cus = device_cu_count();
  RowsPlan best{1, 1};
  double best_t = 1e30;
  for (int gw : {4, 2, 1}) {
    if (ng % gw != 0) continue;
    const long ngb = ng / gw;
    for (int split = 1; split <= std::min(16, ks); ++split) {
      const long wgs = (ngb * split + 3) / 4, rounds = (wgs + cus - 1) / cus;
      const double t = 0.146 * rounds * (gw + 0.25 * mb) * ((ks + split - 1) / split) +
                       2.0 * split * M * (double)N * 4 / 8e6;
      if (t < best_t - 1e-9) {
        best_t = t;
        best = RowsPlan{gw, split};
      }
    }
  }
  return best;
}

// ---- Register-direct weights, activations through LDS (a few hundred rows) --
//
// At a few hundred rows (the batch-1 forward) every tile of the LDS-staged
// kernel above reads both operands out of LDS: a 64 x 96 wave tile moves 160
// bytes of LDS per 64 x 96 x 2 flops per k, near gfx950's LDS/MFMA balance, and
// a third of its issue slots go to the DMA bursts and the per-k-step barrier.
// Here the weights come from their packed copy (each 32-row x 16-k MFMA operand
// one lane-ordered 1 KiB run) straight into a P-slice register ring, so only
// the activation tile is staged: per wave 32 TI bytes of LDS per k against 32
// TI x 32 TJ x 2 flops.  W is the MFMA A operand, the activation rows the B
// operand, so a lane ends with 16 virtual weight rows of one token row: the
// SwiGLU pair (gate, up) and the rotate-half pair (d, d + 64) of an output sit
// in registers r and r + 8 of one lane and the epilogues need no exchange.
//
// Workgroup: 4 waves (one per SIMD).  NWN of them sit side by side along N,
// each owning TJ 32-row groups of Bv; KG = 4 / NWN k-groups split every 64-k
// step (group g takes the 16-k slices g 4/KG .. of it), their accumulators
// added through LDS after the loop.  The activation tile [BM, 64 KSTEPS] of a
// stage streams by LDS-DMA into an AS-stage ring (128-byte rows, swizzled as
// above), one barrier per stage.  Past the last stage the DMA and the weight
// loads are issued again on the last valid addresses (their results are never
// used), so every wait below counts a fixed number of later loads.
template <int TI_, int TJ_, int NWN_, int KSTEPS_, int AS_, int P_, int PF_ = 0>
struct WdTile {
  static constexpr int TI = TI_, TJ = TJ_, NWN = NWN_, KG = 4 / NWN_, KSTEPS = KSTEPS_, AS = AS_, P = P_;
  static constexpr int PF = PF_;  // stages ahead of the L2 prefetch of the weight tile (0: none)
  static constexpr int NW = 4, NTH = 256;
  static constexpr int BM = 32 * TI, BN = 32 * TJ * NWN;
  static constexpr int SPS = 4 * KSTEPS;                // 16-k slices per stage
  static constexpr int SPG = 4 / KG;                    // slices of a 64-k step one k-group takes
  static constexpr int U = SPS / KG;                    // slices per stage one wave computes
  static constexpr int STAGE = BM * 128 * KSTEPS;       // LDS bytes per stage
  static constexpr int IA = BM * KSTEPS / 8 / NW;       // LDS-DMA instructions per wave per stage
  static constexpr int IU = IA / U;                     // ... issued in each of its slices
  static constexpr int R = P > U ? P / U : 1;           // stages unrolled per loop iteration
  static_assert(NWN * KG == 4, "four waves");
  static_assert(BM * KSTEPS % (8 * NW) == 0, "activation rows split evenly over the DMA loads");
  static_assert(IU * U == IA && IU >= 1, "the stage's DMA spreads evenly over the wave's slices");
  static_assert(P % U == 0 || U % P == 0, "register ring slots fixed at compile time");
  static_assert(AS >= 3, "a stage is filled while the one before it is read");
  static_assert(U % 2 == 0, "fragment register sets alternate within a stage");
  // Issue order of a wave in stage s: per slice, IU DMA loads of stage
  // s + AS - 1 (into the slot stage s - 1 left), then (last slice) the wait
  // and barrier, the MFMAs, TJ weight loads for the slice P later.  At the
  // last slice of stage t the wave waits for its DMA of stage t + 1; loads
  // issued after the last of them: the steady count (stage t + 1 issued in
  // stage t + 2 - AS) or the first stages' (stages 1 .. AS - 2 issued before
  // the loop), clamped to vmcnt's range.  And before the loop, the loads after
  // its DMA of stage 0.
  static constexpr int PER = TJ + IU;  // loads per slice
  static constexpr int C1 = TJ + (AS - 3) * U * PER + (U - 1) * PER + IU;
  static constexpr int C0 = (AS - 3) * IA + P * TJ + (U - 1) * PER + IU;
  static constexpr int CMIN = C0 < C1 ? C0 : C1;
  static constexpr int CWAIT = CMIN < 63 ? CMIN : 63;
  static constexpr int CFIRST = ((AS - 2) * IA + P * TJ) < 63 ? (AS - 2) * IA + P * TJ : 63;
  static constexpr size_t LDS = (size_t)AS * STAGE;
  static constexpr size_t MERGE = KG == 1 ? 0 : (size_t)NWN * TI * TJ * 16 * 64 * 4;
  static constexpr size_t LDS_BYTES = LDS > MERGE ? LDS : MERGE;
  static constexpr size_t LDS_ALLOC = LDS_BYTES + 256;  // + the prefetch loads' scratch word per lane
};
// Batch-1 gate/up (M = 512, N = 24576): 4 x 64 = 256 workgroups of 128 x 384
using WdWide = WdTile<4, 3, 4, 2, 4, 8>;
// q/k/v-sized launches: 128 x 192 in two k-groups (M = 512, N = 12288: 256 workgroups)
using WdKg2 = WdTile<4, 3, 2, 2, 4, 8>;
// residual projections (N = d_model): 128 x 256, split over K (M = 512, N =
// 4096: 64 tiles x 4 splits), or 128 x 128 in two k-groups (128 tiles x 2);
// both prefetch their weights two stages ahead into L2 (LLaDA-8B shape at 512
// rows: down 54.0 -> 51.7 us, output projection 26.9 -> 25.6 us; on the
// gate/up and q/k/v tiles the same prefetch halved the L1-miss latency and
// changed nothing, 85.8 / 60.4 us either way)
using WdRes = WdTile<4, 2, 4, 2, 4, 8, 2>;
using WdRes2 = WdTile<4, 2, 2, 2, 4, 8, 2>;
// q/k/v or gate/up launches whose 128 x 192 tiles would leave most CUs idle
// (Dream-7B shape at 768 rows: N = 4608, 216 tiles of 128 x 128 where 128 x
// 192 makes 144): 128 x 128 in two k-groups
using WdQ2 = WdTile<4, 2, 2, 2, 4, 8>;
// gate/up widths that no 192- or 384-wide tile divides (Dream-7B: N = 37888 =
// 148 x 256): 256 x 256 on 4 waves of 256 x 64, one 64-k step per stage (the
// four-stage ring takes 128 KiB of LDS); per flop a quarter fewer bytes per CU
// than 128 x 384, and 256 registers of accumulators per lane
using WdBig = WdTile<8, 2, 4, 1, 4, 8>;

template <class TL, int EPI>
__global__ void __launch_bounds__(256, 1) gemm_wd_kernel(GemmArgs g) {
#if defined(__HIP_DEVICE_COMPILE__)
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int TI = TL::TI, TJ = TL::TJ, U = TL::U, P = TL::P, AS = TL::AS, R = TL::R;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave % TL::NWN, kg = wave / TL::NWN;
  const int MT = (g.M + TL::BM - 1) / TL::BM, T = MT * (g.N / TL::BN), S = (int)gridDim.x / T;
  // XCD x runs workgroups i = x mod 8: it takes a contiguous run of the
  // (K split, N tile, M tile) order, so the M tiles of one weight tile share
  // its L2 and, split, an XCD streams one k-range of the weights (measured:
  // giving each XCD one row tile instead, so that its activations stay in
  // its L2 while the other row tiles re-read the weights from MALL, took the
  // batch-1 gate/up from 89 to 129 us)
  const int i = blockIdx.x, x = i & 7, TS = (int)gridDim.x;
  const int li = x * (TS >> 3) + min(x, TS & 7) + (i >> 3);
  const int tile = li % T, z = li / T;
  const int m0 = (tile % MT) * TL::BM, n0 = (tile / MT) * TL::BN;
  // split z takes the stages [z nst, (z + 1) nst) of K
  const int nk = g.K / 64, nst = nk / TL::KSTEPS / S, st0 = z * nst;

  // activation DMA: instruction q of wave w fills rows 8 (4 q + w) .. +7 of the
  // stage's row space [KSTEPS][BM] (sub-block = row / BM); lane l writes row +
  // l/8, slot l%8, holding the row's chunk (l%8) ^ ((row >> 1) & 7)
  const int lr = lane >> 3, lc = (lane & 7) ^ (((wave & 1) << 2) | (lr >> 1));
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc((void*)g.A, 0, 0x7fffffff, 0x00020000);
  uint32_t voa[TL::IA];
#pragma unroll
  for (int q = 0; q < TL::IA; ++q) {
    const int r = 8 * (4 * q + wave) + lr, sb = r / TL::BM, row = min(m0 + r % TL::BM, g.M - 1);
    voa[q] = (uint32_t)(((size_t)row * g.K + sb * 64 + lc * 8) * 2);
  }
  // DMA instruction q of stage t (past the end: the last stage again, never read)
  auto issue_a = [&](int t, int q) {
    t = min(t, nst - 1);
    char* base = lds + (t % AS) * TL::STAGE;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(base + 8 * (4 * q + wave) * 128), 16, voa[q],
                                             (st0 + t) * TL::KSTEPS * 128, 0, 0);
  };
  // weights: group G = n0 / 32 + wn TJ + j of the packed copy.  The wave's
  // slice uu of stage t is 16-k slice t SPS + 4 (uu / SPG) + kg SPG + uu % SPG.
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc((void*)g.Wp, 0, 0x7fffffff, 0x00020000);
  uint32_t wbase[TJ];
#pragma unroll
  for (int j = 0; j < TJ; ++j) {
    const int G = n0 / 32 + wn * TJ + j;
    wbase[j] = (uint32_t)((((size_t)(G >> 3) * nk * 8 + (G & 7)) * 4) * 1024 + lane * 16 +
                          (kg * TL::SPG) * 1024);
  }
  // L2 prefetch (PF > 0): the MT row tiles that share this weight tile each
  // touch one 128-byte line per lane of their share of its stage PF ahead
  // (dword LDS-DMA loads into a scratch word per lane of LDS: no registers
  // held), so that the weight loads of all of them find the lines in their
  // XCD's L2
  constexpr int NG = TJ * TL::NWN, LPS = NG * 32 * TL::KSTEPS;
  const int LP = (LPS + MT - 1) / MT, NI = (LP + 63) / 64;
  uint32_t pfo[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int pl = min((tile % MT) * LP + min((wave + 4 * q) * 64 + lane, LP - 1), LPS - 1);
    const int ks = pl / (NG * 32), rem = pl % (NG * 32), G = n0 / 32 + rem / 32;
    pfo[q] = (uint32_t)(((size_t)(G >> 3) * nk + ks) * 32768 + (G & 7) * 4096 + (rem % 32) * 128);
  }
  auto prefetch = [&](int t) {
    if (TL::PF == 0 || t >= nst) return;
#pragma unroll
    for (int q = 0; q < 2; ++q)
      if (wave + 4 * q < NI)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)(lds + TL::LDS_BYTES), 4, pfo[q],
                                                 (st0 + t) * (TL::KSTEPS * 32768), 0, 0);
  };
  typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
  u32x4_t wbuf[P][TJ];
  // operand j of the wave's slice uu (compile-time) of stage t, into ring slot
  auto load_w = [&](int t, int uu, int slot, int j) {
    t = min(t, nst - 1);  // past the end: the last stage again, never used
    const uint32_t off =
        (uint32_t)((st0 + t) * (TL::KSTEPS * 32768) + (uu / TL::SPG) * 32768 + (uu % TL::SPG) * 1024);
    wbuf[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(rw, wbase[j] + off, 0, 2);  // non-temporal
  };
  // activation operands of slice uu of the stage in LDS at base
  const int lrow = lane & 31, lhalf = lane >> 5;
  bf16x8_t af[2][TI];
  auto frag = [&](const char* base, int uu, int set) {
    const int sb = uu / TL::SPG, sl = kg * TL::SPG + uu % TL::SPG;
#pragma unroll
    for (int ii = 0; ii < TI; ++ii)
      af[set][ii] = *reinterpret_cast<const bf16x8_t*>(base + sb * TL::BM * 128 + swz(32 * ii + lrow, 2 * sl + lhalf));
  };

  f32x16_t acc[TJ][TI];
#pragma unroll
  for (int j = 0; j < TJ; ++j)
#pragma unroll
    for (int ii = 0; ii < TI; ++ii)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][ii][r] = 0.f;

#pragma unroll
  for (int t = 0; t < AS - 1; ++t)
#pragma unroll
    for (int q = 0; q < TL::IA; ++q) issue_a(t, q);
#pragma unroll
  for (int v = 0; v < P; ++v)
#pragma unroll
    for (int j = 0; j < TJ; ++j) load_w(v / U, v % U, v, j);
  wait_vm_lds<TL::CFIRST>();
  barrier_nofence();
  frag(lds, 0, 0);

  for (int t0 = 0; t0 < nst; t0 += R) {
#pragma unroll
    for (int rr = 0; rr < R; ++rr) {
      const int t = t0 + rr;
      const char* base = lds + (t % AS) * TL::STAGE;
#pragma unroll
      for (int uu = 0; uu < U; ++uu) {
        const int slot = (rr * U + uu) % P;
        // the slice that reuses this ring slot: P slices later
        const int tn = t + (uu + P) / U, un = (uu + P) % U;
        __builtin_amdgcn_sched_barrier(0);
        if (TL::PF > 0 && uu == 0) {
          prefetch(t + TL::PF);
          __builtin_amdgcn_sched_barrier(0);
        }
        // a share of stage t + AS - 1 into the slot stage t - 1 left (every
        // wave passed the barrier that ended it)
#pragma unroll
        for (int q = 0; q < TL::IU; ++q) issue_a(t + AS - 1, uu * TL::IU + q);
        if (uu + 1 < U) {
          frag(base, uu + 1, (uu + 1) & 1);
        } else {
          // this wave's DMA of stage t + 1 has landed once at most CWAIT later
          // loads are outstanding; after the barrier every wave's has, and
          // every wave is done reading stage t
          wait_vm_lds<TL::CWAIT>();
          barrier_nofence();
          frag(lds + ((t + 1) % AS) * TL::STAGE, 0, 0);
        }
        // MFMAs operand-major; each weight operand's slot is refilled right
        // after its last use
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
#pragma unroll
          for (int ii = 0; ii < TI; ++ii)
            acc[j][ii] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wbuf[slot][j]),
                                                                af[uu & 1][ii], acc[j][ii], 0, 0, 0);
          load_w(tn, un, slot, j);
        }
        __builtin_amdgcn_sched_group_barrier(0x020, TL::IU, 0);  // the DMA share
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          if (j == 0) {
#pragma unroll
            for (int ii = 0; ii < TI; ++ii) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // an MFMA
              __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // a fragment read of the next slice
            }
          } else {
            __builtin_amdgcn_sched_group_barrier(0x008, TI, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // the refill of operand j
        }
      }
    }
  }
  wait_vm_lds<0>();
  barrier_nofence();  // the ring is idle

  // With two k-groups the sum of the groups' accumulators is finished by
  // group 0 for the residual epilogue; for the staged ones group 0 finishes
  // row blocks ii < TI / 2 and group 1 the others (each hands the other its
  // share through LDS), so all four waves stage.  Two addends: the same sum
  // in either order.
  constexpr bool SPLIT_ROWS = TL::KG == 2 && EPI != EPI_RESID && TI % 2 == 0;
  auto own_rows = [&](int ii) { return !SPLIT_ROWS ? kg == 0 : (ii < TI / 2) == (kg == 0); };
  if (TL::KG == 2) {
    float4* xa = reinterpret_cast<float4*>(lds) + (size_t)wn * (TI * TJ * 4 * 64) + lane;
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int ii = 0; ii < TI; ++ii) {
        if (own_rows(ii)) continue;  // the share this wave hands over
#pragma unroll
        for (int q = 0; q < 4; ++q)
          xa[((j * TI + ii) * 4 + q) * 64] =
              make_float4(acc[j][ii][4 * q], acc[j][ii][4 * q + 1], acc[j][ii][4 * q + 2], acc[j][ii][4 * q + 3]);
      }
    wait_vm_lds<0>();
    barrier_nofence();
    // the second group joins the staged epilogues' barriers and stores
    if (kg == 1 && EPI == EPI_RESID) return;
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int ii = 0; ii < TI; ++ii) {
        if (!own_rows(ii)) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 v = xa[((j * TI + ii) * 4 + q) * 64];
          acc[j][ii][4 * q] += v.x;
          acc[j][ii][4 * q + 1] += v.y;
          acc[j][ii][4 * q + 2] += v.z;
          acc[j][ii][4 * q + 3] += v.w;
        }
      }
  }

  // Epilogue.  Lane l holds, for token row m = m0 + 32 ii + l % 32 and group G,
  // virtual rows 32 G + 8 (r / 4) + 4 (l / 32) + r % 4 in register r.
  constexpr int HD = 128, HALF = 64;
  const int nq = g.Hq * HD, nkv = g.Hkv * HD;
  const float inv_l = 1.0f / (float)g.Lq;
  bool v_over = false;
  if constexpr (EPI == EPI_SWIGLU || EPI == EPI_QKV_ROPE) {
    // 16-bit outputs go through LDS (the ring is idle) in the destination's
    // order and leave as 16-byte stores of the whole workgroup (StageGeo, as
    // in the LDS-staged kernel); written from the MFMA layout they were
    // 8-byte pieces of 32 rows per instruction, and v^T 2-byte stores
    using St = StageGeo<TL::BM, TL::BN>;
    static_assert((EPI == EPI_SWIGLU ? St::SW_BYTES : St::QKV_BYTES) <= (int)TL::LDS_BYTES, "staging fits the ring");
    wait_vm_lds<0>();
    barrier_nofence();  // every wave is done reading the ring (and the k-group merge area)
    {
#pragma unroll
      for (int ii = 0; ii < TI; ++ii) {
        if (!own_rows(ii)) continue;
        const int ml = 32 * ii + lrow, m = m0 + ml;  // rows past M are never staged nor stored
        if (m >= g.M) continue;
        int p = 0;
        if (EPI == EPI_QKV_ROPE) p = seq_pos(m, g.Lq, inv_l).y;
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          const int jb = wn * TJ + j, G = n0 / 32 + jb;
          const f32x16_t& a = acc[j][ii];
          char* blk = lds + jb * St::BLK;
          if (EPI == EPI_SWIGLU) {
            // registers 0..7: gate of tile column 16 jb + 8 (r / 4) + 4 (l / 32) + r % 4, r + 8: its up
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              float o[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float gt = a[4 * q + e], up = a[4 * q + 8 + e];
                o[e] = __fdividef(gt, 1.0f + __expf(-gt)) * up;
              }
              *reinterpret_cast<uint2*>(lds + ml * St::SW_ROW + (16 * jb + 8 * q + 4 * lhalf) * 2) =
                  make_uint2(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]));
            }
          } else if (32 * G < nq + nkv) {
            // q or k: registers 0..7 dimension d = 16 blk + 8 (r / 4) + 4 (l / 32) + r % 4 of the
            // head, r + 8: d + 64; the block's row holds d0 .. d0 + 15, then d0 + 64 .. d0 + 79
            const int rel = 32 * G < nq ? 32 * G : 32 * G - nq, bk = (rel % HD) >> 5, pos = g.pos0 + p;
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              const int d = 16 * bk + 8 * q + 4 * lhalf;
              const float4 c4 = *reinterpret_cast<const float4*>(g.cosb + (size_t)pos * HALF + d);
              const float4 s4 = *reinterpret_cast<const float4*>(g.sinb + (size_t)pos * HALF + d);
              const float cc[4] = {c4.x, c4.y, c4.z, c4.w}, ss[4] = {s4.x, s4.y, s4.z, s4.w};
              float lo[4], hi[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float x1 = a[4 * q + e], x2 = a[4 * q + 8 + e];
                lo[e] = x1 * cc[e] - x2 * ss[e];
                hi[e] = x2 * cc[e] + x1 * ss[e];
              }
              *reinterpret_cast<uint2*>(blk + ml * 64 + (8 * q + 4 * lhalf) * 2) =
                  make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
              *reinterpret_cast<uint2*>(blk + ml * 64 + (16 + 8 * q + 4 * lhalf) * 2) =
                  make_uint2(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]));
            }
          } else {
            // v: register r is channel 8 (r / 4) + 4 (l / 32) + r % 4 of the block, staged as v^T
#pragma unroll
            for (int r = 0; r < 16; ++r)
              *reinterpret_cast<f16_t*>(blk + (8 * (r >> 2) + 4 * lhalf + (r & 3)) * St::VROW + ml * 2) =
                  v_half(a[r], v_over);
          }
        }
      }
    }
    __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
    barrier_nofence();
    staged_store<TL::BM, TL::BN, TL::NTH, EPI>(g, lds, m0, n0);
    if (EPI == EPI_QKV_ROPE && v_over && g.err) atomicOr(g.err, (int)ERR_V_RANGE);
    return;
  }
  // residual projections: float32 results straight from the MFMA layout
#pragma unroll
  for (int ii = 0; ii < TI; ++ii) {
    const int m = m0 + 32 * ii + lrow;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int G = n0 / 32 + wn * TJ + j;
      const f32x16_t& a = acc[j][ii];
      if (S > 1) {  // split over K: partial z [M, N] float32, summed in z order later
        float* part = g.splitk_buf + (size_t)z * g.M * g.N + (size_t)m * g.N + 32 * G + 4 * lhalf;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<float4*>(part + 8 * q) = make_float4(a[4 * q], a[4 * q + 1], a[4 * q + 2], a[4 * q + 3]);
      } else {  // h[m, n] += result, n = 32 G + 8 q + 4 (l / 32) + e
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float4* hp = reinterpret_cast<float4*>(g.resid + (size_t)m * g.N + 32 * G + 8 * q + 4 * lhalf);
          float4 h = *hp;
          h.x += a[4 * q];
          h.y += a[4 * q + 1];
          h.z += a[4 * q + 2];
          h.w += a[4 * q + 3];
          *hp = h;
        }
      }
    }
  }
#endif
}

// Register-direct-weight plan for a launch of 129 .. 1024 rows with the packed
// copy (tile 0: none, 1: WdWide, 2: WdKg2, 3: WdRes, 4: WdRes2, 5: WdQ2; split over K),
// taken when the tile's workgroups fill at least 7/8 of the rounds they take
// on the compute units.  At these sizes a workgroup is bounded by the bytes
// its CU pulls through the vector-memory path, (BM + BN) x its k-range x 2
// (the texture-address unit ~80% busy on the gate/up launch), so the time
// model is rounds x (20.4 us per MB + 5 us), calibrated on the LLaDA-8B shape
// at 512 rows (gate/up WdWide 85.6 us, q/k/v WdKg2 59.3, down WdRes at split 4
// 54.9, output projection WdRes2 at split 2 26.1, down WdRes2 at split 2
// 60.9), plus for split-K the partials the next norm reads (~1.5 us per split
// per 2^21 outputs: the fused norm at 512 x 4096 took 7.6 / 10.6 / 14.6 us
// with 2 / 4 / 8 of them); a split's k-range must be whole stages of at
// least 2048 k.  Elsewhere the LDS-staged tiles stay.
struct WdPlan {
  int tile, split;
};
WdPlan wd_plan(int M, int N, int K, int epi) {
  WdPlan best{0, 1};
  if (M <= 128 || M > 1024 || K % 64 != 0) return best;
  const int nk = K / 64;
  const long cus = device_cu_count();
  double best_t = 1e30;
  // fill16: the least sixteenths of the rounds' workgroup slots the tiles must fill
  auto consider = [&](int id, int BM, int BN, int KSTEPS, int R, int split, bool one_round = false,
                      int fill16 = 14) {
    if (N % BN != 0 || nk % (KSTEPS * split) != 0 || (nk / KSTEPS / split) % R != 0) return;
    const long T = (long)((M + BM - 1) / BM) * (N / BN) * split, rounds = (T + cus - 1) / cus;
    if (one_round ? (rounds > 1 || 4 * T < 3 * cus) : 16 * T < fill16 * rounds * cus) return;
    double t = (double)rounds * (20.4e-6 * (BM + BN) * (double)(K / split) * 2 + 5.0);
    if (split > 1) t += 1.5 * split * (double)M * N / (1 << 21);
    if (t < best_t - 1e-9) {
      best_t = t;
      best = WdPlan{id, split};
    }
  };
  if (epi == EPI_SWIGLU || epi == EPI_QKV_ROPE) {
    consider(1, WdWide::BM, WdWide::BN, WdWide::KSTEPS, WdWide::R, 1);
    // 256 x 256 also at 13/16 of its rounds' slots (Dream-7B gate/up at 768
    // rows: 444 tiles), where no other register-direct tile divides N
    if (epi == EPI_SWIGLU) consider(6, WdBig::BM, WdBig::BN, WdBig::KSTEPS, WdBig::R, 1, false, 13);
    consider(2, WdKg2::BM, WdKg2::BN, WdKg2::KSTEPS, WdKg2::R, 1);
    // 128 x 128 when its tiles take one round on at least three quarters of
    // the CUs: the LDS-staged tiles fill no more of them at these widths (over
    // several rounds the wider LDS-staged tiles pull fewer bytes per CU)
    consider(5, WdQ2::BM, WdQ2::BN, WdQ2::KSTEPS, WdQ2::R, 1, true);
  } else if (epi == EPI_RESID) {
    // only splits of at least 2048 k: the output projection at 512 rows (K =
    // 4096, split 4) ran 27 us + 9.9 us for its partials in the norm against
    // 26.4 + 8.1 on the LDS-staged 128 x 128 tile at split 2; the down
    // projection (K = 12288, split 4) 54.9 + 9.9 against 52.5 + 14.6 at split 8
    for (int split = 1; split <= 8 && K / split >= 2048; ++split) {
      consider(3, WdRes::BM, WdRes::BN, WdRes::KSTEPS, WdRes::R, split);
      consider(4, WdRes2::BM, WdRes2::BN, WdRes2::KSTEPS, WdRes2::R, split);
    }
  }
  return best;
}

struct Plan {
  int bm, bn, kg, split;
};

// Pick the tile and a K split (any count up to 8, or 16 for launches of at most
// 128 rows; the k-steps are spread as evenly as they divide), by a time model:
// rounds of workgroups over the 256 compute units x k-steps per workgroup x
// the tile's k-step time (measured on random bf16 data at M = 512: larger
// tiles move fewer LDS bytes per flop and run two waves per SIMD), plus, for
// the residual GEMMs, the memory time of the float32 partials (written here,
// read back by the reduction) or of the residual's read-modify-write, at the
// ~8 TB/s they move at (measured: much of it stays in the last-level cache).
// Only residual GEMMs split at more than 128 rows; at most 128 rows (the block
// rows of a cached step) the q/k/v and SwiGLU GEMMs split too, their epilogues
// then running on the summed partials, and the 64-row tile is a candidate.  A
// launch is also bounded by streaming its weights from HBM once.  The 192-wide
// tiles exist for the widths where 256-wide tiles leave CUs idle (batch-1
// q/k/v and gate/up).
Plan plan(int M, int N, int K, int epi) {
  struct Cand {
    int bm, bn, kg;
    double t_kstep_us;
  };
  const Cand cands[] = {{128, 256, 1, 1.04}, {256, 256, 1, 1.71}, {256, 192, 1, 1.37}, {128, 192, 1, 0.87},
                        {128, 192, 2, 0.81}, {64, 256, 2, 0.55}, {128, 128, 2, 0.46}};
  constexpr double BYTES_PER_US = 8.0e6;
  // the weights stream from HBM once per launch (tiles of one N range share
  // them through L2) at ~6.5 TB/s when every CU has a workgroup
  constexpr double W_BYTES_PER_US = 6.5e6;
  Plan best{0, 0, 0, 0};
  double best_t = 1e30;
  const int ksteps = K / BK;
  for (const Cand& c : cands) {
    if (N % c.bn != 0 || (c.bm == 64 && M > 128)) continue;
    const long tiles = (long)((M + c.bm - 1) / c.bm) * (N / c.bn);
    // the 128 x 128 tile only where it measured faster: output projections
    // (K <= 4096) of 160 .. 512 rows -- LLaDA-8B shape at 512 rows 29.5 + 8.8
    // us for the GEMM and its reduction at split 2 against 33.4 + 11.3 for
    // 128 x 256 at split 4, 23.4 against 26.2 us at 160 rows; it lost on the
    // down projections (longer K) and at 768 rows (51.3 against 48.2 us) --
    // and q/k/v launches whose 128 x 128 tiles fit one round on the CUs
    // (Dream-7B shape at 768 rows: 216 tiles, 46 against 57 us for 144 tiles
    // of 128 x 192; at 384 tiles, LLaDA-8B at 512 rows, it lost: 95 against 72)
    if (c.bn == 128 && !(M > 128 && ((epi == EPI_RESID && K <= 4096 && M <= 512) ||
                                     (epi == EPI_QKV_ROPE && tiles <= 256))))
      continue;
    const int max_split = M <= 128 ? 16 : 8;
    for (int split = 1; split <= max_split; ++split) {
      if (split > 1 && ((epi != EPI_RESID && M > 128) || ksteps / split < 4)) break;
      const long rounds = (tiles * split + 255) / 256;
      const double t_mma = (double)rounds * ((ksteps + split - 1) / split) * c.t_kstep_us;
      const double t_w = 2.0 * N * K / (W_BYTES_PER_US * std::min(1.0, (double)(tiles * split) / 256));
      // at a few dozen rows the weight stream bounds every tile; the tile's own
      // k-step time still shows through (only partly hidden under the stream)
      double t = std::max(t_mma, t_w);
      if (M <= 128) t += 0.25 * std::min(t_mma, t_w);
      if (epi == EPI_RESID || split > 1) t += 8.0 * split * (double)M * N / BYTES_PER_US;
      if (t < best_t - 1e-9) {
        best_t = t;
        best = Plan{c.bm, c.bn, c.kg, split};
      }
    }
  }
  if (best.bm == 0) throw HipError("gemm_bf16: N must be a multiple of 192 or 256");
  return best;
}

template <class TL, int EPI, bool PB = false>
void launch_tile(const GemmArgs& g, int split, hipStream_t s) {
  const int tiles = ((g.M + TL::BM - 1) / TL::BM) * (g.N / TL::BN);
  const size_t lds = lds_bytes<TL, EPI>();
  static const hipError_t attr = hipFuncSetAttribute((const void*)gemm_bf16_kernel<TL, EPI, PB>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hip_check(attr, "hipFuncSetAttribute(gemm_bf16)");
  hipLaunchKernelGGL((gemm_bf16_kernel<TL, EPI, PB>), dim3(tiles, 1, split), dim3(TL::NTH), lds, s, g);
}

template <int EPI>
void launch_epi(const GemmArgs& g, const Plan& p, hipStream_t s) {
  if (p.bm == 64 && g.Wp)
    launch_tile<TileT, EPI, true>(g, p.split, s);
  else if (p.bm == 64)
    launch_tile<TileT, EPI>(g, p.split, s);
  else if (p.bm == 128 && p.bn == 128)
    launch_tile<TileQ, EPI>(g, p.split, s);
  else if (p.bm == 256 && p.bn == 256)
    launch_tile<TileL, EPI>(g, p.split, s);
  else if (p.bm == 256)
    launch_tile<TileM, EPI>(g, p.split, s);
  else if (p.bn == 256)
    launch_tile<TileS, EPI>(g, p.split, s);
  else
    p.kg == 2 ? launch_tile<TileSM2, EPI>(g, p.split, s) : launch_tile<TileSM, EPI>(g, p.split, s);
}

}  // namespace

size_t gemm_packed_bytes(int N, int K) { return (size_t)ceil_div(N, 256) * 256 * (size_t)K * sizeof(bf16_t); }

void launch_pack_gemm_weights(const GemmArgs& g, bf16_t* out, hipStream_t s) {
  if (g.K % BK != 0) throw HipError("pack_gemm_weights: K % 64 must be 0");
  if (gemm_packed_bytes(g.N, g.K) > 0x7fffffffu) throw HipError("pack_gemm_weights: matrix larger than 2 GiB");
  const size_t nvec = gemm_packed_bytes(g.N, g.K) / 16;
  const int grid = (int)std::min<size_t>(ceil_div(nvec, (size_t)256), 8192);
  switch (g.epi) {
    case EPI_QKV_ROPE: hipLaunchKernelGGL(pack_gemm_weights_kernel<EPI_QKV_ROPE>, dim3(grid), dim3(256), 0, s, g, out, nvec); break;
    case EPI_SWIGLU: hipLaunchKernelGGL(pack_gemm_weights_kernel<EPI_SWIGLU>, dim3(grid), dim3(256), 0, s, g, out, nvec); break;
    default: hipLaunchKernelGGL(pack_gemm_weights_kernel<EPI_RESID>, dim3(grid), dim3(256), 0, s, g, out, nvec); break;
  }
  DLLM_LAUNCH_CHECK("pack_gemm_weights");
}

// launches the register-direct kernel can take (given the packed copy)
bool rows_path(int M, int N, int K) { return M >= 1 && M <= 64 && N % 32 == 0 && K % 64 == 0; }

size_t gemm_bf16_splitk_bytes(int M, int N, int K, int epi) {
  const Plan p = plan(M, N, K, epi);
  size_t b = p.split > 1 ? (size_t)p.split * M * N * sizeof(float) : 0;
  const WdPlan wp = wd_plan(M, N, K, epi);  // with packed weights
  if (wp.tile && wp.split > 1) b = std::max(b, (size_t)wp.split * M * N * sizeof(float));
  if (rows_path(M, N, K)) b = std::max(b, (size_t)rows_plan(M, N, K).split * M * N * sizeof(float));
  return b;
}

template <int S>
void launch_splitk_resid(const float* part, float* resid, long MN, hipStream_t s) {
  hipLaunchKernelGGL(splitk_resid_kernel<S>, dim3(ceil_div(MN / 4, 256)), dim3(256), 0, s, part, resid, MN);
}

// The register-direct path: partials from gemm_rows_kernel, then the epilogue.
// A residual GEMM's partials are left to the next norm when defer is given
// (its 1024-thread fused kernel adds them), else reduced across the chip.
void launch_gemm_rows(const GemmArgs& a, hipStream_t s, PendingResid* defer) {
  const RowsPlan rp = rows_plan(a.M, a.N, a.K);
  RowsArgs r{a.A, a.Wp, a.splitk_buf, a.M, a.N, a.K, rp.split, a.N / 32 / rp.gw};
  const dim3 grid(ceil_div(r.ngb * r.S, 4)), blk(256);
  const bool two = a.M > 32;
  auto go = [&](auto gwc) {
    constexpr int GW = decltype(gwc)::value;
    if (two)
      hipLaunchKernelGGL((gemm_rows_kernel<GW, 2, 4>), grid, blk, 0, s, r);
    else
      hipLaunchKernelGGL((gemm_rows_kernel<GW, 1, 8>), grid, blk, 0, s, r);
  };
  if (rp.gw == 4)
    go(std::integral_constant<int, 4>{});
  else if (rp.gw == 2)
    go(std::integral_constant<int, 2>{});
  else
    go(std::integral_constant<int, 1>{});
  DLLM_LAUNCH_CHECK("gemm_rows");
  if (a.epi == EPI_SWIGLU) {
    const long n = (long)a.M * (a.N / 2);
    hipLaunchKernelGGL(splitk_swiglu_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, a.splitk_buf, rp.split, a.M,
                       a.N / 2, a.out);
  } else if (a.epi == EPI_QKV_ROPE) {
    const long n = (long)a.M * a.N;
    hipLaunchKernelGGL(splitk_qkv_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, a.splitk_buf, rp.split, a);
  } else if (defer && a.M <= RESID_NORM_WIDE_ROWS) {
    *defer = PendingResid{a.splitk_buf, rp.split};
  } else {
    const long MN = (long)a.M * a.N;
    switch (rp.split) {
#define DLLM_CASE(S_) \
  case S_: launch_splitk_resid<S_>(a.splitk_buf, a.resid, MN, s); break;
      DLLM_CASE(1) DLLM_CASE(2) DLLM_CASE(3) DLLM_CASE(4) DLLM_CASE(5) DLLM_CASE(6) DLLM_CASE(7) DLLM_CASE(8)
      DLLM_CASE(9) DLLM_CASE(10) DLLM_CASE(11) DLLM_CASE(12) DLLM_CASE(13) DLLM_CASE(14) DLLM_CASE(15) DLLM_CASE(16)
#undef DLLM_CASE
      default: throw HipError("gemm_rows: split must be 1 .. 16");
    }
  }
  DLLM_LAUNCH_CHECK("gemm_rows epilogue");
}

template <class TL, int EPI>
void launch_wd_tile(const GemmArgs& g, int split, hipStream_t s) {
  const int T = ((g.M + TL::BM - 1) / TL::BM) * (g.N / TL::BN);
  static const hipError_t attr = hipFuncSetAttribute((const void*)gemm_wd_kernel<TL, EPI>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)TL::LDS_ALLOC);
  hip_check(attr, "hipFuncSetAttribute(gemm_wd)");
  hipLaunchKernelGGL((gemm_wd_kernel<TL, EPI>), dim3(T * split), dim3(TL::NTH), TL::LDS_ALLOC, s, g);
}


void launch_gemm_bf16(const GemmArgs& a, hipStream_t s, PendingResid* defer) {
  if (defer) *defer = PendingResid{};
  if (a.M == 0) return;
  if (a.K % BK != 0) throw HipError("gemm_bf16: K % 64 must be 0");
  if (a.epi == EPI_QKV_ROPE && (a.n0 % 128 != 0 || a.n1 % 128 != 0))
    throw HipError("gemm_bf16: q and k/v regions must be whole 128-row heads");
  if (a.epi == EPI_QKV_ROPE && (a.M >= (1 << 24) || a.B >= (1 << 16)))
    throw HipError("gemm_bf16: q/k/v epilogue needs B * L < 2^24 and B < 2^16");
  if (a.epi == EPI_QKV_ROPE && (a.Lq < 1 || a.pos0 < 0 || a.pos0 + a.Lq > a.L || a.M % a.Lq != 0))
    throw HipError("gemm_bf16: q/k/v rows must be whole windows of Lq positions inside the sequence");
  if (a.Wp && rows_path(a.M, a.N, a.K)) {  // few rows from the packed copy: register-direct
    launch_gemm_rows(a, s, defer);
    return;
  }
  const WdPlan wp = a.Wp ? wd_plan(a.M, a.N, a.K, a.epi) : WdPlan{0, 1};
  if (wp.tile) {  // a few hundred rows: register-direct weights, staged activations
    if (wp.tile == 1)
      a.epi == EPI_SWIGLU ? launch_wd_tile<WdWide, EPI_SWIGLU>(a, 1, s) : launch_wd_tile<WdWide, EPI_QKV_ROPE>(a, 1, s);
    else if (wp.tile == 2)
      a.epi == EPI_SWIGLU ? launch_wd_tile<WdKg2, EPI_SWIGLU>(a, 1, s) : launch_wd_tile<WdKg2, EPI_QKV_ROPE>(a, 1, s);
    else if (wp.tile == 5)
      a.epi == EPI_SWIGLU ? launch_wd_tile<WdQ2, EPI_SWIGLU>(a, 1, s) : launch_wd_tile<WdQ2, EPI_QKV_ROPE>(a, 1, s);
    else if (wp.tile == 6)
      launch_wd_tile<WdBig, EPI_SWIGLU>(a, 1, s);
    else if (wp.tile == 3)
      launch_wd_tile<WdRes, EPI_RESID>(a, wp.split, s);
    else
      launch_wd_tile<WdRes2, EPI_RESID>(a, wp.split, s);
    DLLM_LAUNCH_CHECK("gemm_wd");
    if (wp.split > 1 && defer) {
      *defer = PendingResid{a.splitk_buf, wp.split};  // the next norm adds them
    } else if (wp.split > 1) {
      const long MN = (long)a.M * a.N;
      switch (wp.split) {
#define DLLM_CASE(S_) \
  case S_: launch_splitk_resid<S_>(a.splitk_buf, a.resid, MN, s); break;
        DLLM_CASE(2) DLLM_CASE(3) DLLM_CASE(4) DLLM_CASE(5) DLLM_CASE(6) DLLM_CASE(7) DLLM_CASE(8)
#undef DLLM_CASE
        default: throw HipError("gemm_wd: split must be 1 .. 8");
      }
      DLLM_LAUNCH_CHECK("splitk_resid");
    }
    return;
  }
  const Plan p = plan(a.M, a.N, a.K, a.epi);
  switch (a.epi) {
    case EPI_QKV_ROPE: launch_epi<EPI_QKV_ROPE>(a, p, s); break;
    case EPI_SWIGLU: launch_epi<EPI_SWIGLU>(a, p, s); break;
    case EPI_RESID: launch_epi<EPI_RESID>(a, p, s); break;
    default: throw HipError("gemm_bf16: unknown epilogue");
  }
  DLLM_LAUNCH_CHECK("gemm_bf16");
  if (p.split > 1 && a.epi == EPI_SWIGLU) {
    const long n = (long)a.M * (a.N / 2);
    hipLaunchKernelGGL(splitk_swiglu_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, a.splitk_buf, p.split, a.M,
                       a.N / 2, a.out);
    DLLM_LAUNCH_CHECK("splitk_swiglu");
  } else if (p.split > 1 && a.epi == EPI_QKV_ROPE) {
    const long n = (long)a.M * a.N;
    hipLaunchKernelGGL(splitk_qkv_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, a.splitk_buf, p.split, a);
    DLLM_LAUNCH_CHECK("splitk_qkv");
  } else if (p.split > 1 && defer && a.M > 128) {
    // few rows (M <= 128) are reduced right away across the whole chip: the
    // fused reduce + norm runs one workgroup per row
    *defer = PendingResid{a.splitk_buf, p.split};
  } else if (p.split > 1) {
    const long MN = (long)a.M * a.N;
    const dim3 grid(ceil_div(MN / 4, 256));
    auto go = [&](auto sc) {
      hipLaunchKernelGGL(splitk_resid_kernel<decltype(sc)::value>, grid, dim3(256), 0, s, a.splitk_buf, a.resid, MN);
    };
    switch (p.split) {
      case 2: go(std::integral_constant<int, 2>{}); break;
      case 3: go(std::integral_constant<int, 3>{}); break;
      case 4: go(std::integral_constant<int, 4>{}); break;
      case 5: go(std::integral_constant<int, 5>{}); break;
      case 6: go(std::integral_constant<int, 6>{}); break;
      case 7: go(std::integral_constant<int, 7>{}); break;
      case 8: go(std::integral_constant<int, 8>{}); break;
      case 9: go(std::integral_constant<int, 9>{}); break;
      case 10: go(std::integral_constant<int, 10>{}); break;
      case 11: go(std::integral_constant<int, 11>{}); break;
      case 12: go(std::integral_constant<int, 12>{}); break;
      case 13: go(std::integral_constant<int, 13>{}); break;
      case 14: go(std::integral_constant<int, 14>{}); break;
      case 15: go(std::integral_constant<int, 15>{}); break;
      case 16: go(std::integral_constant<int, 16>{}); break;
      default: throw HipError("splitk_resid: split must be 2 .. 16");
    }
    DLLM_LAUNCH_CHECK("splitk_resid");
  }
}

}  // namespace dllm
