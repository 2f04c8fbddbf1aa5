// Embedding gather, RoPE table, RMSNorm and decoding-state initialisation.
#include "kernels.h"

#include <type_traits>

namespace dllm {

int device_cu_count() {
  static const int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    return n;
  }();
  return cus;
}

// One 256-thread block per row; every thread converts a strided set of columns.
// Row m = b rows + i gathers token x[b, row0 + i]; an id outside [0, V) is
// never used as an address: the row is zero and the error word says so.
template <typename T>
__global__ void __launch_bounds__(256) embed_kernel(const int32_t* __restrict__ x, const T* __restrict__ E,
                                                    float* __restrict__ h, int rows, int L, int row0, int d, int V,
                                                    int* __restrict__ err, int* __restrict__ zero, int nzero) {
  const int m = blockIdx.x, b = m / rows, i = m - b * rows;
  if (m == 0)
    for (int z = threadIdx.x; z < nzero; z += 256) zero[z] = 0;
  const int tok = x[(size_t)b * L + row0 + i];
  const bool ok = tok >= 0 && tok < V;
  const size_t src = (size_t)(ok ? tok : 0) * d;
  float* dst = h + (size_t)m * d;
  for (int c = threadIdx.x; c < d; c += 256) dst[c] = ok ? Act<T>::load(E, src + c) : 0.f;
  if (!ok && threadIdx.x == 0 && err) atomicOr(err, (int)ERR_TOKEN_RANGE);
}

void launch_embed(const int32_t* x, const void* E, int dtype, float* h, int B, int rows, int L, int row0, int d,
                  int V, int* err, hipStream_t s, int* zero, int nzero) {
  const int M = B * rows;
  if (M == 0) return;
  if (!zero) nzero = 0;
  if (dtype == 0)
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, s, x, (const float*)E, h, rows, L, row0, d, V,
                       err, zero, nzero);
  else
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(M), dim3(256), 0, s, x, (const bf16_t*)E, h, rows, L, row0, d, V,
                       err, zero, nzero);
  DLLM_LAUNCH_CHECK("embed");
}

// angle = pos * base^(-2j/hd) in float64 (positions reach 8k, where a float32
// angle would already be off by ~1e-3 rad), stored as float32 cos/sin.  Thread
// 0 also clears the forward's error word (err non-null).
__global__ void rope_table_kernel(float* cosb, float* sinb, int L, int half, double base, int hd, int* err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0 && err) *err = 0;
  if (i >= L * half) return;
  const int pos = i / half, j = i % half;
  const double inv_freq = pow(base, -2.0 * (double)j / (double)hd);
  double sn, cs;
  sincos((double)pos * inv_freq, &sn, &cs);
  cosb[i] = (float)cs;
  sinb[i] = (float)sn;
}

void launch_rope_table(float* cosb, float* sinb, int L, int hd, double base, int* err, hipStream_t s) {
  const int n = L * (hd / 2);
  if (n == 0) return;
  hipLaunchKernelGGL(rope_table_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, cosb, sinb, L, hd / 2, base, hd,
                     err);
  DLLM_LAUNCH_CHECK("rope_table");
}

// RMSNorm of one row per 256-thread block.  The sum of squares is accumulated
// in float64 in a fixed order (per-thread strided sums, then a fixed tree), so
// results are run-to-run identical; scaling and the gain are applied in float32.
template <typename TG, typename TO>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const float* __restrict__ h, const TG* __restrict__ g,
                                                      TO* __restrict__ out, int rows, int L, int row0, int d,
                                                      float eps) {
  const int r = blockIdx.x;
  const int b = r / rows, i = r % rows;
  const float* src = h + ((size_t)b * L + row0 + i) * d;
  double ss = 0.0;
  for (int c = threadIdx.x; c < d; c += 256) {
    const double v = src[c];
    ss += v * v;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  __shared__ double part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  const double tot = (part[0] + part[1]) + (part[2] + part[3]);
  const float rstd = (float)(1.0 / sqrt(tot / (double)d + (double)eps));
  TO* dst = out + (size_t)r * d;
  for (int c = threadIdx.x; c < d; c += 256) Act<TO>::store(dst, c, src[c] * rstd * Act<TG>::load(g, c));
}

// Vector form of the same computation for d % 4 == 0 and d <= 1024 NV: the
// row is read once, as float4, into registers (NV per thread) and written from
// there.  The float64 sum of squares runs over a different fixed order; its
// float32 result is the same in all but astronomically rare ties.
template <typename T> struct Vec4;
template <> struct Vec4<float> {
  static __device__ __forceinline__ float4 load(const float* p, int c4) { return reinterpret_cast<const float4*>(p)[c4]; }
  static __device__ __forceinline__ void store(float* p, int c4, float4 v) { reinterpret_cast<float4*>(p)[c4] = v; }
};
template <> struct Vec4<bf16_t> {
  static __device__ __forceinline__ float4 load(const bf16_t* p, int c4) {
    const uint2 u = reinterpret_cast<const uint2*>(p)[c4];
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
  }
  static __device__ __forceinline__ void store(bf16_t* p, int c4, float4 v) {
    uint2 u;
    u.x = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
    u.y = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
    reinterpret_cast<uint2*>(p)[c4] = u;
  }
};

template <typename TG, typename TO, int NV>
__global__ void __launch_bounds__(256) rmsnorm_vec_kernel(const float* __restrict__ h, const TG* __restrict__ g,
                                                          TO* __restrict__ out, int rows, int L, int row0, int d,
                                                          float eps) {
  const int r = blockIdx.x;
  const int b = r / rows, i = r % rows;
  const float* src = h + ((size_t)b * L + row0 + i) * d;
  const int d4 = d / 4;
  float4 v[NV];
  double ss = 0.0;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = threadIdx.x + 256 * j;
    if (c < d4) {
      v[j] = Vec4<float>::load(src, c);
      ss += (double)v[j].x * v[j].x + (double)v[j].y * v[j].y + (double)v[j].z * v[j].z + (double)v[j].w * v[j].w;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  __shared__ double part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  const double tot = (part[0] + part[1]) + (part[2] + part[3]);
  const float rstd = (float)(1.0 / sqrt(tot / (double)d + (double)eps));
  TO* dst = out + (size_t)r * d;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = threadIdx.x + 256 * j;
    if (c < d4) {
      const float4 gg = Vec4<TG>::load(g, c);
      Vec4<TO>::store(dst, c,
                      make_float4(v[j].x * rstd * gg.x, v[j].y * rstd * gg.y, v[j].z * rstd * gg.z, v[j].w * rstd * gg.w));
    }
  }
}

template <typename TG, typename TO>
void launch_rmsnorm_t(const float* h, const TG* g, TO* out, int B, int rows, int L, int row0, int d, float eps,
                      hipStream_t s) {
  const dim3 grid(B * rows), blk(256);
  const bool aligned = ((uintptr_t)h | (uintptr_t)g | (uintptr_t)out) % 16 == 0;
  if (d % 4 == 0 && aligned && d <= 1024 * 8) {
    const int nv = ceil_div(d, 1024);
    if (nv <= 2)
      hipLaunchKernelGGL((rmsnorm_vec_kernel<TG, TO, 2>), grid, blk, 0, s, h, g, out, rows, L, row0, d, eps);
    else if (nv <= 4)
      hipLaunchKernelGGL((rmsnorm_vec_kernel<TG, TO, 4>), grid, blk, 0, s, h, g, out, rows, L, row0, d, eps);
    else
      hipLaunchKernelGGL((rmsnorm_vec_kernel<TG, TO, 8>), grid, blk, 0, s, h, g, out, rows, L, row0, d, eps);
  } else {
    hipLaunchKernelGGL((rmsnorm_kernel<TG, TO>), grid, blk, 0, s, h, g, out, rows, L, row0, d, eps);
  }
}

// rmsnorm_vec_kernel preceded by the split-K residual update of its row: each
// float4 of the row is h + ((p_0 + p_1) + ... + p_{S-1}), the same operations in
// the same order as splitk_resid_kernel, written back to h and kept for the norm.
// NT threads per row: 256, or 1024 for a few rows (a cached step's block
// rows, whose register-direct GEMMs leave up to 16 partials): one workgroup per
// row then has every partial load of the row in flight at once.
template <int NV, int S, int NT = 256>
__global__ void __launch_bounds__(NT) resid_rmsnorm_kernel(float* __restrict__ h, const float* __restrict__ part,
                                                           long MN, const bf16_t* __restrict__ g,
                                                           bf16_t* __restrict__ out, int d, float eps) {
  const int r = blockIdx.x;
  float* row = h + (size_t)r * d;
  const int d4 = d / 4;
  float4 v[NV];
  double ss = 0.0;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = threadIdx.x + NT * j;
    if (c < d4) {
      const size_t i = (size_t)r * d4 + c;
      float4 acc = reinterpret_cast<const float4*>(part)[i];
#pragma unroll
      for (int z = 1; z < S; ++z) {
        const float4 p = reinterpret_cast<const float4*>(part + (size_t)z * MN)[i];
        acc.x += p.x;
        acc.y += p.y;
        acc.z += p.z;
        acc.w += p.w;
      }
      float4 x = Vec4<float>::load(row, c);
      x.x += acc.x;
      x.y += acc.y;
      x.z += acc.z;
      x.w += acc.w;
      Vec4<float>::store(row, c, x);
      v[j] = x;
      ss += (double)x.x * x.x + (double)x.y * x.y + (double)x.z * x.z + (double)x.w * x.w;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  constexpr int NWV = NT / 64;
  __shared__ double prt[NWV];
  if ((threadIdx.x & 63) == 0) prt[threadIdx.x >> 6] = ss;
  __syncthreads();
  double tot = 0.0;
  if (NWV == 4) {
    tot = (prt[0] + prt[1]) + (prt[2] + prt[3]);
  } else {
#pragma unroll
    for (int w = 0; w < NWV; ++w) tot += prt[w];
  }
  const float rstd = (float)(1.0 / sqrt(tot / (double)d + (double)eps));
  bf16_t* dst = out + (size_t)r * d;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = threadIdx.x + NT * j;
    if (c < d4) {
      const float4 gg = Vec4<bf16_t>::load(g, c);
      Vec4<bf16_t>::store(dst, c, make_float4(v[j].x * rstd * gg.x, v[j].y * rstd * gg.y, v[j].z * rstd * gg.z,
                                              v[j].w * rstd * gg.w));
    }
  }
}

void launch_resid_rmsnorm(float* h, const PendingResid& pend, const bf16_t* g, bf16_t* out, int M, int d, float eps,
                          hipStream_t s) {
  if (M == 0) return;
  if (d % 4 != 0 || d > 8192 || ((uintptr_t)h | (uintptr_t)pend.part | (uintptr_t)g | (uintptr_t)out) % 16 != 0)
    throw HipError("resid_rmsnorm: needs d % 4 == 0, d <= 8192 and 16-byte aligned rows");
  const long MN = (long)M * d;
  // the split count is a template parameter so that every partial's loads are in flight at once
  if (M <= RESID_NORM_WIDE_ROWS) {
    auto go = [&](auto nvc, auto sc) {
      hipLaunchKernelGGL((resid_rmsnorm_kernel<decltype(nvc)::value, decltype(sc)::value, 1024>), dim3(M), dim3(1024),
                         0, s, h, pend.part, MN, g, out, d, eps);
    };
    auto by_split = [&](auto nvc) {
      switch (pend.split) {
#define DLLM_CASE(S_) \
  case S_: go(nvc, std::integral_constant<int, S_>{}); break;
        DLLM_CASE(1) DLLM_CASE(2) DLLM_CASE(3) DLLM_CASE(4) DLLM_CASE(5) DLLM_CASE(6) DLLM_CASE(7) DLLM_CASE(8)
        DLLM_CASE(9) DLLM_CASE(10) DLLM_CASE(11) DLLM_CASE(12) DLLM_CASE(13) DLLM_CASE(14) DLLM_CASE(15)
        DLLM_CASE(16)
#undef DLLM_CASE
        default: throw HipError("resid_rmsnorm: split must be 1 .. 16");
      }
    };
    if (d <= 4096)
      by_split(std::integral_constant<int, 1>{});
    else
      by_split(std::integral_constant<int, 2>{});
    DLLM_LAUNCH_CHECK("resid_rmsnorm");
    return;
  }
  const int nv = ceil_div(d, 1024);
  auto go = [&](auto nvc, auto sc) {
    hipLaunchKernelGGL((resid_rmsnorm_kernel<decltype(nvc)::value, decltype(sc)::value>), dim3(M), dim3(256), 0, s, h,
                       pend.part, MN, g, out, d, eps);
  };
  auto by_split = [&](auto nvc) {
    switch (pend.split) {
      case 2: go(nvc, std::integral_constant<int, 2>{}); break;
      case 3: go(nvc, std::integral_constant<int, 3>{}); break;
      case 4: go(nvc, std::integral_constant<int, 4>{}); break;
      case 5: go(nvc, std::integral_constant<int, 5>{}); break;
      case 6: go(nvc, std::integral_constant<int, 6>{}); break;
      case 7: go(nvc, std::integral_constant<int, 7>{}); break;
      case 8: go(nvc, std::integral_constant<int, 8>{}); break;
      default: throw HipError("resid_rmsnorm: split must be 2 .. 8");
    }
  };
  if (nv <= 2)
    by_split(std::integral_constant<int, 2>{});
  else if (nv <= 4)
    by_split(std::integral_constant<int, 4>{});
  else
    by_split(std::integral_constant<int, 8>{});
  DLLM_LAUNCH_CHECK("resid_rmsnorm");
}

// rmsnorm_vec_kernel for the bf16 head rows, also writing the rows in MFMA
// B-operand order (row r < 32, columns 4c .. 4c+3 are eight contiguous bytes:
// slice c / 4, lane r + 32 ((c / 2) % 2), elements 4 (c % 2) ..).  With S > 0
// split-K partials [S, MN] pending from the last residual GEMM, each float4 of
// the row is first h + ((p_0 + p_1) + ... + p_{S-1}) (splitk_resid_kernel's
// operations and order), written back to h.  Block 0 also zeroes the LM
// head's ticket.
template <int NV>
__global__ void __launch_bounds__(256) rmsnorm_head_kernel(float* __restrict__ h, const float* __restrict__ part,
                                                           int S, long MN, const bf16_t* __restrict__ g,
                                                           bf16_t* __restrict__ out, bf16_t* __restrict__ outf,
                                                           int rows, int L, int row0, int d, float eps,
                                                           int* __restrict__ ticket) {
  const int r = blockIdx.x;
  const int b = r / rows, i = r % rows;
  const size_t hrow = (size_t)b * L + row0 + i;
  float* src = h + hrow * d;
  const int d4 = d / 4;
  if (ticket && r == 0 && threadIdx.x == 0) *ticket = 0;
  float4 v[NV];
  double ss = 0.0;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = threadIdx.x + 256 * j;
    if (c < d4) {
      v[j] = Vec4<float>::load(src, c);
      if (S > 0) {
        const size_t pi = hrow * d4 + c;
        float4 acc = reinterpret_cast<const float4*>(part)[pi];
#pragma unroll 4
        for (int z = 1; z < S; ++z) {
          const float4 p = reinterpret_cast<const float4*>(part + (size_t)z * MN)[pi];
          acc.x += p.x;
          acc.y += p.y;
          acc.z += p.z;
          acc.w += p.w;
        }
        v[j].x += acc.x;
        v[j].y += acc.y;
        v[j].z += acc.z;
        v[j].w += acc.w;
        Vec4<float>::store(src, c, v[j]);
      }
      ss += (double)v[j].x * v[j].x + (double)v[j].y * v[j].y + (double)v[j].z * v[j].z + (double)v[j].w * v[j].w;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  __shared__ double wsum[4];
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = ss;
  __syncthreads();
  const double tot = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
  const float rstd = (float)(1.0 / sqrt(tot / (double)d + (double)eps));
  bf16_t* dst = out + (size_t)r * d;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int c = threadIdx.x + 256 * j;
    if (c < d4) {
      const float4 gg = Vec4<bf16_t>::load(g, c);
      const float4 y = make_float4(v[j].x * rstd * gg.x, v[j].y * rstd * gg.y, v[j].z * rstd * gg.z,
                                   v[j].w * rstd * gg.w);
      Vec4<bf16_t>::store(dst, c, y);
      if (outf) Vec4<bf16_t>::store(outf, ((size_t)(c >> 2) * 64 + r + 32 * ((c >> 1) & 1)) * 2 + (c & 1), y);
    }
  }
}

void launch_rmsnorm_head(float* h, const PendingResid* pend, const bf16_t* g, bf16_t* out, bf16_t* outf, int B,
                         int rows, int L, int row0, int d, float eps, int* ticket, hipStream_t s) {
  if (B * rows == 0) return;
  const float* part = pend && pend->split > 0 ? pend->part : nullptr;
  const int S = part ? pend->split : 0;
  if (d % 4 != 0 || d > 8192 ||
      ((uintptr_t)h | (uintptr_t)g | (uintptr_t)out | (uintptr_t)outf | (uintptr_t)part) % 16 != 0)
    throw HipError("rmsnorm_head: needs d % 4 == 0, d <= 8192 and 16-byte aligned rows");
  if (outf && B * rows > HEAD_FRAG_ROWS) throw HipError("rmsnorm_head: operand-order copy holds 32 rows");
  const long MN = (long)B * L * d;
  const int nv = ceil_div(d, 1024);
  const dim3 grid(B * rows), blk(256);
  if (nv <= 2)
    hipLaunchKernelGGL(rmsnorm_head_kernel<2>, grid, blk, 0, s, h, part, S, MN, g, out, outf, rows, L, row0, d, eps,
                       ticket);
  else if (nv <= 4)
    hipLaunchKernelGGL(rmsnorm_head_kernel<4>, grid, blk, 0, s, h, part, S, MN, g, out, outf, rows, L, row0, d, eps,
                       ticket);
  else
    hipLaunchKernelGGL(rmsnorm_head_kernel<8>, grid, blk, 0, s, h, part, S, MN, g, out, outf, rows, L, row0, d, eps,
                       ticket);
  DLLM_LAUNCH_CHECK("rmsnorm_head");
}

void launch_rmsnorm(const float* h, const void* g, void* out, int dtype, int B, int rows, int L, int row0, int d,
                    float eps, hipStream_t s) {
  if (B * rows == 0) return;
  if (dtype == 0)
    launch_rmsnorm_t(h, (const float*)g, (float*)out, B, rows, L, row0, d, eps, s);
  else
    launch_rmsnorm_t(h, (const bf16_t*)g, (bf16_t*)out, B, rows, L, row0, d, eps, s);
  DLLM_LAUNCH_CHECK("rmsnorm");
}

__global__ void state_init_kernel(const int32_t* __restrict__ prompt, int32_t* __restrict__ x,
                                  int32_t* __restrict__ commit_step, int8_t* __restrict__ reason,
                                  float* __restrict__ sv, int32_t* __restrict__ budget, int32_t* __restrict__ ell,
                                  int32_t* __restrict__ done, int B, int P, int G, int mask_id,
                                  int* __restrict__ err) {
  const int L = P + G;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0 && err) *err = 0;
  if (i < B * L) {
    const int b = i / L, l = i % L;
    x[i] = l < P ? prompt[(size_t)b * P + l] : mask_id;
  }
  if (i < B * G) {
    commit_step[i] = -1;
    reason[i] = 0;
    sv[i] = 0.f;
    budget[i] = 0;
  }
  if (i < B) {
    ell[i] = 0;
    done[i] = 0;
  }
}

void launch_state_init(const int32_t* prompt, int32_t* x, int32_t* commit_step, int8_t* reason, float* sv,
                       int32_t* budget, int32_t* ell, int32_t* done, int B, int P, int G, int mask_id,
                       int* err, hipStream_t s) {
  const int n = B * (P + G);
  if (n == 0) return;
  hipLaunchKernelGGL(state_init_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, prompt, x, commit_step, reason,
                     sv, budget, ell, done, B, P, G, mask_id, err);
  DLLM_LAUNCH_CHECK("state_init");
}

}  // namespace dllm
