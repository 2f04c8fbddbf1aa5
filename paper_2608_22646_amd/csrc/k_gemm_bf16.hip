// bf16 GEMM on CDNA4 matrix cores with the step's fused epilogues.
//
//   C[M, N] = A[M, K] * Bv[N, K]^T       (both operands K-contiguous, fp32 accumulate)
//
// Bv is a "virtual" weight matrix whose rows come from up to three tensors, so
// q/k/v and gate/up never need to be concatenated in memory:
//   QKV    : rows [0, n0) of Wq, then n1 rows of Wk, then Wv; the epilogue applies
//            rotate-half RoPE to q and k and writes q [B,Hq,L,hd], k [B,Hkv,L,hd]
//            as bf16 and v^T [B,Hkv,hd,L] as the bf16-rounded values in IEEE half.
//   SWIGLU : 32-row chunks alternate between Wgate and Wup (gate rows f..f+31, then
//            up rows f..f+31), so one lane holds gate and up of the same column f;
//            the epilogue writes silu(gate) * up as bf16 [M, F].
//   RESID  : plain W; the epilogue adds the result to the float32 residual.
//
// Tiling: 128 x 256 x 64 per 256-thread workgroup, 2 x 2 wavefronts, each wave owns
// a 64 x 128 block of 32x32 MFMA tiles (v_mfma_f32_32x32x16_bf16).  Tiles of A and
// Bv stream from memory straight into a 3-stage LDS ring (buffer_load_dwordx4 ...
// lds, no staging registers): two k-tiles are in flight while the third is
// consumed, with one barrier per k-step.  LDS rows are 128 bytes (64 bf16); the
// 16-byte chunk c of row r is stored at slot c ^ (r & 7), so the eight rows read
// by eight consecutive lanes hit eight different bank groups.
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

// Virtual weight row n -> (tensor index, row inside that tensor).  QKV regions
// are whole 256-row tiles (Hq and Hkv even), so a tile reads a single tensor;
// SwiGLU rows interleave gate and up every 32 rows.
template <int EPI>
__device__ __forceinline__ int2 vrow(const GemmArgs& g, int n) {
  if (EPI == EPI_QKV_ROPE) {
    if (n < g.n0) return make_int2(0, n);
    if (n < g.n0 + g.n1) return make_int2(1, n - g.n0);
    return make_int2(2, n - g.n0 - g.n1);
  }
  if (EPI == EPI_SWIGLU) {
    const int chunk = n >> 5;
    return make_int2(chunk & 1, ((chunk >> 1) << 5) + (n & 31));
  }
  return make_int2(0, n);
}

__device__ __forceinline__ int swz(int row, int chunk) { return row * 128 + ((chunk ^ (row & 7)) << 4); }

template <int BM_, int BN_, int WAVES_M, int WAVES_N, int STAGES_>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, S = STAGES_;
  static constexpr int NW = WAVES_M * WAVES_N, NTH = 64 * NW;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int TI = WM / 32, TJ = WN / 32;          // MFMA tiles per wave
  static constexpr int IA = BM / 8 / NW, IB = BN / 8 / NW;   // LDS-DMA instructions per wave per stage
  static constexpr int LDS_STAGE = (BM + BN) * 128;
  static_assert(WN == 128, "the QKV and SwiGLU epilogues need 128-column wave tiles");
  static_assert(IA * NW * 8 == BM && IB * NW * 8 == BN, "tile rows must split evenly over the DMA loads");
};
// 128 x 256, 4 waves of 64 x 128, three stages (small M: more tiles to spread over 256 CUs)
using TileS = Tile<128, 256, 2, 2, 3>;
// 256 x 256, 8 waves of 64 x 128 (two per SIMD), two stages (large M: fewer bytes per flop)
using TileL = Tile<256, 256, 4, 2, 2>;

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Wait until at most N of this wave's vector-memory operations are in flight
// (gfx9 s_waitcnt encoding: vmcnt split over bits 3:0 and 15:14, expcnt and
// lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
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

template <class TL, int EPI>
__global__ void __launch_bounds__(TL::NTH, 1) gemm_bf16_kernel(GemmArgs g) {
  // The buffer-resource builtins exist only for the device target; the host
  // pass needs just the kernel's signature for its launch stub.
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int BM = TL::BM, BN = TL::BN, S = TL::S, NW = TL::NW;
  extern __shared__ __attribute__((aligned(16))) char lds[];
  // wave index made provably uniform so per-wave buffer descriptors stay scalar
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / (BN / TL::WN), wn = wave % (BN / TL::WN);

  // XCD-aware, grouped tile order.  Workgroup i runs on XCD i % 8, so each XCD
  // takes a contiguous run of the tile order; the order walks groups of up to
  // GM M-tiles across all N-tiles, so the ~32 tiles an XCD runs at once share
  // a few A tiles and a few weight tiles in that XCD's L2.
  constexpr int GM = 8;
  const int mt = (g.M + BM - 1) / BM, ntl = g.N / BN;
  const int tiles = mt * ntl;
  int lin = blockIdx.x;
  if ((tiles & 7) == 0) lin = (blockIdx.x & 7) * (tiles >> 3) + (blockIdx.x >> 3);
  const int grp = lin / (GM * ntl), first_m = grp * GM, gsize = min(mt - first_m, GM);
  const int in_grp = lin - grp * GM * ntl;
  const int m0 = (first_m + in_grp % gsize) * BM, n0 = (in_grp / gsize) * BN;

  const int ksplit = g.K / gridDim.z;
  const int kbeg = blockIdx.z * ksplit;
  const int nk = ksplit / BK;

  // LDS-DMA loads: instruction i of wave w fills tile rows 8 (NW i + w) .. +7
  // (1 KiB of LDS).  Lane l writes row + l/8, slot l%8, which holds the row's
  // logical 16-byte chunk (l%8) ^ (l/8) (the XOR swizzle, since row % 8 == l/8).
  // Row offsets are fixed across k; the k advance goes in the scalar offset.
  // A rows past M are clamped to M-1 (their results are never stored).
  const int lr = lane >> 3, lc = (lane & 7) ^ (lane >> 3);
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc((void*)g.A, 0, 0x7fffffff, 0x00020000);
  uint32_t voa[TL::IA];
#pragma unroll
  for (int i = 0; i < TL::IA; ++i) {
    const int row = min(m0 + 8 * (NW * i + wave) + lr, g.M - 1);
    voa[i] = (uint32_t)(((size_t)row * g.K + kbeg + lc * 8) * 2);
  }
  // Bv rows: each 8-row DMA group lies in one tensor (the tile's q/k/v tensor,
  // or gate / up by 32-row parity for SwiGLU).
  const bf16_t* wsrc[3] = {g.W0, g.W1, g.W2};
  __amdgpu_buffer_rsrc_t rbs[TL::IB];
  uint32_t vob[TL::IB];
#pragma unroll
  for (int i = 0; i < TL::IB; ++i) {
    const int2 first = vrow<EPI>(g, n0 + 8 * (NW * i + wave));  // wave-uniform
    rbs[i] = __builtin_amdgcn_make_buffer_rsrc((void*)wsrc[first.x], 0, 0x7fffffff, 0x00020000);
    vob[i] = (uint32_t)(((size_t)(first.y + lr) * g.K + kbeg + lc * 8) * 2);
  }
  auto issue = [&](int kt) {
    char* base = lds + (kt % S) * TL::LDS_STAGE;
    const int soff = kt * BK * 2;
#pragma unroll
    for (int i = 0; i < TL::IA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(base + 8 * (NW * i + wave) * 128), 16, voa[i], soff,
                                               0, 0);
#pragma unroll
    for (int i = 0; i < TL::IB; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rbs[i], (lds_ptr_t)(base + BM * 128 + 8 * (NW * i + wave) * 128), 16,
                                               vob[i], soff, 0, 0);
  };

  f32x16_t acc[TL::TI][TL::TJ];
#pragma unroll
  for (int i = 0; i < TL::TI; ++i)
#pragma unroll
    for (int j = 0; j < TL::TJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  constexpr int PER_STAGE = TL::IA + TL::IB;  // DMA instructions per wave per stage
#pragma unroll
  for (int s = 0; s < S - 1; ++s)
    if (s < nk) issue(s);

  const int lrow = lane & 31, lhalf = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    // tile kt has landed once only the later tiles' loads are outstanding
    if (kt + 1 < nk)
      wait_vmcnt<PER_STAGE * (S - 2)>();
    else
      wait_vmcnt<0>();
    barrier_nofence();  // tile kt visible to all waves; stage (kt - 1) % S free
    if (kt + S - 1 < nk) issue(kt + S - 1);
    const char* base = lds + (kt % S) * TL::LDS_STAGE;
    // Software pipeline over the four 16-wide k-slices: slices 0 and 1 are read
    // first, then each MFMA of slice ks is followed by one LDS read of slice
    // ks + 2 (three fragment register sets), so LDS latency hides under the
    // MFMAs.  The sched_group_barrier sequence pins that order.
    constexpr int NS = BK / 16, NF = TL::TI + TL::TJ, NM = TL::TI * TL::TJ;
    static_assert(NM >= NF, "pipeline needs at least as many MFMAs as fragment reads per slice");
    bf16x8_t af[3][TL::TI], bfr[3][TL::TJ];
    auto frag = [&](int ks) {
      const int ch = ks * 2 + lhalf, set = ks % 3;
#pragma unroll
      for (int i = 0; i < TL::TI; ++i)
        af[set][i] = *reinterpret_cast<const bf16x8_t*>(base + swz(wm * TL::WM + i * 32 + lrow, ch));
#pragma unroll
      for (int j = 0; j < TL::TJ; ++j)
        bfr[set][j] = *reinterpret_cast<const bf16x8_t*>(base + BM * 128 + swz(wn * TL::WN + j * 32 + lrow, ch));
    };
    frag(0);
    frag(1);
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * NF, 0);
#pragma unroll
    for (int ks = 0; ks < NS; ++ks) {
      if (ks + 2 < NS) frag(ks + 2);
#pragma unroll
      for (int i = 0; i < TL::TI; ++i)
#pragma unroll
        for (int j = 0; j < TL::TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks % 3][i], bfr[ks % 3][j], acc[i][j], 0, 0, 0);
      if (ks + 2 < NS) {
#pragma unroll
        for (int x = 0; x < NF; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA of slice ks
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read of slice ks + 2
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM - NF, 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
      }
    }
  }

  // ------------------------------------------------------------ epilogues
  const int col_in = lane & 31;
  auto row_of = [&](int i, int r) { return m0 + wm * TL::WM + i * 32 + 8 * (r >> 2) + 4 * lhalf + (r & 3); };

  if (gridDim.z > 1) {  // split-K partial tile
    float* part = g.splitk_buf + (size_t)blockIdx.z * g.M * g.N;
#pragma unroll
    for (int i = 0; i < TL::TI; ++i)
#pragma unroll
      for (int j = 0; j < TL::TJ; ++j) {
        const int n = n0 + wn * TL::WN + j * 32 + col_in;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = row_of(i, r);
          if (m < g.M) part[(size_t)m * g.N + n] = acc[i][j][r];
        }
      }
    return;
  }

  if (EPI == EPI_RESID || EPI == EPI_STORE) {
#pragma unroll
    for (int i = 0; i < TL::TI; ++i)
#pragma unroll
      for (int j = 0; j < TL::TJ; ++j) {
        const int n = n0 + wn * TL::WN + j * 32 + col_in;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = row_of(i, r);
          if (m >= g.M) continue;
          if (EPI == EPI_RESID)
            g.resid[(size_t)m * g.N + n] += acc[i][j][r];
          else
            g.out[(size_t)m * g.N + n] = f2bf(acc[i][j][r]);
        }
      }
    return;
  }

  if (EPI == EPI_SWIGLU) {
    const int F = g.N / 2;
#pragma unroll
    for (int i = 0; i < TL::TI; ++i)
#pragma unroll
      for (int j = 0; j < TL::TJ; j += 2) {
        const int chunk = (n0 + wn * TL::WN + j * 32) >> 5;  // even: gate, odd (j+1): up
        const int f = ((chunk >> 1) << 5) + col_in;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = row_of(i, r);
          if (m >= g.M) continue;
          const float gt = acc[i][j][r], up = acc[i][j + 1][r];
          g.out[(size_t)m * F + f] = f2bf(gt / (1.0f + expf(-gt)) * up);
        }
      }
    return;
  }

  // EPI_QKV_ROPE: this wave's 128 columns are exactly one head (hd = 128).
  if (EPI == EPI_QKV_ROPE) {
    constexpr int HD = 128, HALF = 64;
    const int ncol0 = n0 + wn * TL::WN;  // multiple of 128
    const int nq = g.Hq * HD, nk_ = g.Hkv * HD;
    static_assert(TL::TJ == 4, "QKV epilogue needs 128-column wave tiles");
    if (ncol0 < nq + nk_) {
      const bool isq = ncol0 < nq;
      const int head = isq ? ncol0 / HD : (ncol0 - nq) / HD;
      const int H = isq ? g.Hq : g.Hkv;
      bf16_t* dst = isq ? g.q : g.k;
#pragma unroll
      for (int i = 0; i < TL::TI; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int jj = j * 32 + col_in;  // < 64: pairs with jj + 64 (register tile j + 2)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = row_of(i, r);
            if (m >= g.M) continue;
            const int b = m / g.L, pos = m - b * g.L;
            const float c = g.cosb[(size_t)pos * HALF + jj], sn = g.sinb[(size_t)pos * HALF + jj];
            const float x1 = acc[i][j][r], x2 = acc[i][j + 2][r];
            bf16_t* o = dst + (((size_t)b * H + head) * g.L + pos) * HD;
            o[jj] = f2bf(x1 * c - x2 * sn);
            o[jj + HALF] = f2bf(x2 * c + x1 * sn);
          }
        }
    } else {
      const int head = (ncol0 - nq - nk_) / HD;
#pragma unroll
      for (int i = 0; i < TL::TI; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int cj = j * 32 + col_in;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = row_of(i, r);
            if (m >= g.M) continue;
            const int b = m / g.L, pos = m - b * g.L;
            // v is a bf16 value; it is stored as IEEE half (exact in half's range)
            // for the half-precision P.V product of the attention kernel
            g.vt[(((size_t)b * g.Hkv + head) * HD + cj) * g.L + pos] = f2h(bf2f(f2bf(acc[i][j][r])));
          }
        }
    }
  }
#endif
}

// resid[m, n] += sum_z part[z, m, n], z in order.
__global__ void splitk_resid_kernel(const float* __restrict__ part, float* __restrict__ resid, long MN, int S) {
  const long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= MN) return;
  float4 acc = *reinterpret_cast<const float4*>(part + i);
  for (int z = 1; z < S; ++z) {
    const float4 v = *reinterpret_cast<const float4*>(part + (size_t)z * MN + i);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  float4 h = *reinterpret_cast<float4*>(resid + i);
  h.x += acc.x; h.y += acc.y; h.z += acc.z; h.w += acc.w;
  *reinterpret_cast<float4*>(resid + i) = h;
}

struct Plan {
  int bm, bn, split;
};

// Pick the tile (128 x 256 on 4 waves or 256 x 256 on 8 waves) and, for the
// residual GEMMs, a K split, by the number of rounds of workgroups over the
// 256 compute units weighted by each tile's measured per-CU throughput
// (the larger tile moves fewer bytes per flop: ~1.3x faster per flop).
Plan plan(int M, int N, int K, int epi) {
  const double rel_speed[2] = {1.0, 1.3};
  const int bms[2] = {128, 256};
  Plan best{128, 256, 1};
  double best_cost = 1e30;
  for (int c = 0; c < 2; ++c) {
    const long tiles = (long)((M + bms[c] - 1) / bms[c]) * (N / 256);
    int split = 1;
    if (epi == EPI_RESID) {
      while (split < 8 && tiles * split * 2 <= 256 + 64 && (K / BK) % (split * 2) == 0 && (K / BK) / (split * 2) >= 4)
        split *= 2;
    }
    const long wgs = tiles * split;
    const double rounds = (double)((wgs + 255) / 256);
    const double cost = rounds * (double)bms[c] / split / rel_speed[c];
    if (cost < best_cost - 1e-9) {
      best_cost = cost;
      best = Plan{bms[c], 256, split};
    }
  }
  return best;
}

template <class TL, int EPI>
void launch_tile(const GemmArgs& g, int split, hipStream_t s) {
  const int tiles = ((g.M + TL::BM - 1) / TL::BM) * (g.N / TL::BN);
  const size_t lds = (size_t)TL::S * TL::LDS_STAGE;
  static const hipError_t attr = hipFuncSetAttribute((const void*)gemm_bf16_kernel<TL, EPI>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hip_check(attr, "hipFuncSetAttribute(gemm_bf16)");
  hipLaunchKernelGGL((gemm_bf16_kernel<TL, EPI>), dim3(tiles, 1, split), dim3(TL::NTH), lds, s, g);
}

template <int EPI>
void launch_epi(const GemmArgs& g, int bm, int split, hipStream_t s) {
  if (bm == 256)
    launch_tile<TileL, EPI>(g, split, s);
  else
    launch_tile<TileS, EPI>(g, split, s);
}

}  // namespace

size_t gemm_bf16_splitk_bytes(int M, int N, int K, int epi) {
  const Plan p = plan(M, N, K, epi);
  return p.split > 1 ? (size_t)p.split * M * N * sizeof(float) : 0;
}

void launch_gemm_bf16(const GemmArgs& a, hipStream_t s) {
  if (a.M == 0) return;
  if (a.N % 256 != 0 || a.K % BK != 0) throw HipError("gemm_bf16: N % 256 and K % 64 must be 0");
  if (a.epi == EPI_QKV_ROPE && (a.n0 % 256 != 0 || a.n1 % 256 != 0))
    throw HipError("gemm_bf16: q and k/v regions must be multiples of 256 rows");
  const Plan p = plan(a.M, a.N, a.K, a.epi);
  switch (a.epi) {
    case EPI_QKV_ROPE: launch_epi<EPI_QKV_ROPE>(a, p.bm, p.split, s); break;
    case EPI_SWIGLU: launch_epi<EPI_SWIGLU>(a, p.bm, p.split, s); break;
    case EPI_RESID: launch_epi<EPI_RESID>(a, p.bm, p.split, s); break;
    default: throw HipError("gemm_bf16: unknown epilogue");
  }
  DLLM_LAUNCH_CHECK("gemm_bf16");
  if (p.split > 1) {
    const long MN = (long)a.M * a.N;
    hipLaunchKernelGGL(splitk_resid_kernel, dim3(ceil_div(MN / 4, 256)), dim3(256), 0, s, a.splitk_buf, a.resid, MN,
                       p.split);
    DLLM_LAUNCH_CHECK("splitk_resid");
  }
}

}  // namespace dllm
