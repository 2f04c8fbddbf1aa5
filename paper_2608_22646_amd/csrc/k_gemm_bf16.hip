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
// Tiling: BM x BN x 64 per 256-thread workgroup, 2 x 2 wavefronts, each wave owns a
// (BM/2) x (BN/2) block of 32x32 MFMA tiles (v_mfma_f32_32x32x16_bf16).  Tiles of A
// and Bv go global -> registers -> LDS (double buffered, one barrier per k-step).
// LDS rows are 128 bytes (64 bf16); the 16-byte chunk c of row r is stored at slot
// c ^ (r & 7), so the eight rows read by eight consecutive lanes hit eight
// different bank groups.
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
constexpr int NT = 256;

// Source of virtual weight row n for the tile's loads.  QKV regions are whole
// 256-row tiles (Hq and Hkv even), so a tile reads a single tensor; SwiGLU
// tiles interleave gate and up every 32 rows.
template <int EPI>
__device__ __forceinline__ const bf16_t* vrow_ptr(const GemmArgs& g, int n) {
  if (EPI == EPI_QKV_ROPE) {
    if (n < g.n0) return g.W0 + (size_t)n * g.K;
    n -= g.n0;
    if (n < g.n1) return g.W1 + (size_t)n * g.K;
    return g.W2 + (size_t)(n - g.n1) * g.K;
  }
  if (EPI == EPI_SWIGLU) {
    const int chunk = n >> 5;
    const int f = ((chunk >> 1) << 5) + (n & 31);
    return ((chunk & 1) ? g.W1 : g.W0) + (size_t)f * g.K;
  }
  return g.W0 + (size_t)n * g.K;
}

__device__ __forceinline__ int swz(int row, int chunk) { return row * 128 + ((chunk ^ (row & 7)) << 4); }

template <int BM, int BN>
struct Tile {
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int TI = WM / 32, TJ = WN / 32;         // MFMA tiles per wave
  static constexpr int LA = BM * 8 / NT, LB = BN * 8 / NT; // 16-byte loads per thread per stage
  static constexpr int LDS_STAGE = (BM + BN) * 128;
};

template <int BM, int BN, int EPI>
__global__ void __launch_bounds__(NT, 1) gemm_bf16_kernel(GemmArgs g) {
  using TL = Tile<BM, BN>;
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // XCD-aware tile order: workgroup i runs on XCD i % 8; give each XCD a
  // contiguous run of tiles (all M-tiles of consecutive N-tiles) so the weight
  // tile is fetched from HBM once per XCD and A stays in that XCD's L2.
  const int mt = (g.M + BM - 1) / BM, ntl = g.N / BN;
  const int tiles = mt * ntl;
  int lin = blockIdx.x;
  if ((tiles & 7) == 0) lin = (blockIdx.x & 7) * (tiles >> 3) + (blockIdx.x >> 3);
  const int m0 = (lin % mt) * BM, n0 = (lin / mt) * BN;

  const int ksplit = g.K / gridDim.z;
  const int kbeg = blockIdx.z * ksplit;
  const int nk = ksplit / BK;

  // Load e = tid + 256 i covers tile row tid/8 + 32 i, 16-byte chunk tid % 8.
  // Row r of A advances by 32 rows per i; virtual rows of Bv advance by 32 rows
  // per i in the same tensor, except SwiGLU tiles where odd i come from Wup.
  const int lrow0 = tid >> 3, lch = tid & 7;
  const size_t rstride = (size_t)32 * g.K;
  const bf16_t* asrc = g.A + (size_t)min(m0 + lrow0, g.M - 1) * g.K + kbeg + lch * 8;
  const int a_rows_left = g.M - m0 - lrow0;  // load i is valid iff 32 i < a_rows_left
  const bf16_t* bsrc0 = vrow_ptr<EPI>(g, n0 + lrow0) + kbeg + lch * 8;
  const bf16_t* bsrc1 = EPI == EPI_SWIGLU ? vrow_ptr<EPI>(g, n0 + 32 + lrow0) + kbeg + lch * 8 : bsrc0;
  const int st_base = swz(lrow0, lch);  // LDS offset of load i: st_base + i * 32 * 128 (row & 7 unchanged)

  f32x16_t acc[TL::TI][TL::TJ];
#pragma unroll
  for (int i = 0; i < TL::TI; ++i)
#pragma unroll
    for (int j = 0; j < TL::TJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  uint4 ra[TL::LA], rb[TL::LB];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < TL::LA; ++i)
      ra[i] = (32 * i < a_rows_left) ? *reinterpret_cast<const uint4*>(asrc + i * rstride + kt * BK)
                                     : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < TL::LB; ++i) {
      const bf16_t* src = EPI == EPI_SWIGLU ? ((i & 1) ? bsrc1 + (i >> 1) * rstride : bsrc0 + (i >> 1) * rstride)
                                            : bsrc0 + i * rstride;
      rb[i] = *reinterpret_cast<const uint4*>(src + kt * BK);
    }
  };
  auto sstore = [&](int buf) {
    char* base = lds + buf * TL::LDS_STAGE;
#pragma unroll
    for (int i = 0; i < TL::LA; ++i) *reinterpret_cast<uint4*>(base + st_base + i * 32 * 128) = ra[i];
#pragma unroll
    for (int i = 0; i < TL::LB; ++i) *reinterpret_cast<uint4*>(base + BM * 128 + st_base + i * 32 * 128) = rb[i];
  };

  gload(0);
  sstore(0);
  __syncthreads();

  const int lrow = lane & 31, lhalf = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const char* base = lds + buf * TL::LDS_STAGE;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = ks * 2 + lhalf;
      bf16x8_t af[TL::TI], bfr[TL::TJ];
#pragma unroll
      for (int i = 0; i < TL::TI; ++i) {
        const int row = wm * TL::WM + i * 32 + lrow;
        af[i] = *reinterpret_cast<const bf16x8_t*>(base + swz(row, ch));
      }
#pragma unroll
      for (int j = 0; j < TL::TJ; ++j) {
        const int row = wn * TL::WN + j * 32 + lrow;
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(base + BM * 128 + swz(row, ch));
      }
#pragma unroll
      for (int i = 0; i < TL::TI; ++i)
#pragma unroll
        for (int j = 0; j < TL::TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
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

Plan plan(int M, int N, int K, int epi) {
  Plan p{M >= 2048 ? 256 : 128, 256, 1};
  const long tiles = (long)((M + p.bm - 1) / p.bm) * (N / p.bn);
  if (epi == EPI_RESID) {
    while (p.split < 8 && tiles * p.split * 2 <= 256 + 64 && (K / BK) % (p.split * 2) == 0 &&
           (K / BK) / (p.split * 2) >= 4)
      p.split *= 2;
  }
  return p;
}

template <int BM, int BN, int EPI>
void launch_tile(const GemmArgs& g, int split, hipStream_t s) {
  const int tiles = ((g.M + BM - 1) / BM) * (g.N / BN);
  const size_t lds = 2 * (size_t)Tile<BM, BN>::LDS_STAGE;
  static const hipError_t attr = hipFuncSetAttribute((const void*)gemm_bf16_kernel<BM, BN, EPI>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hip_check(attr, "hipFuncSetAttribute(gemm_bf16)");
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, EPI>), dim3(tiles, 1, split), dim3(NT), lds, s, g);
}

template <int EPI>
void launch_epi(const GemmArgs& g, int bm, int split, hipStream_t s) {
  if (bm == 256)
    launch_tile<256, 256, EPI>(g, split, s);
  else
    launch_tile<128, 256, EPI>(g, split, s);
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
