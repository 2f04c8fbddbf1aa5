// float32 path: used by fp32 models (small shapes, where launch latency, not
// arithmetic, bounds the step).  Plain LDS-tiled kernels that keep float32
// storage but accumulate products and softmax sums in float64 (cheap at these
// sizes), so each stored value is the float32 rounding of a nearly exact
// result; fixed reduction order everywhere, so results are run-to-run identical.
#include <algorithm>

#include "kernels.h"

namespace dllm {

// C[M, N] (+)= A[M, K] W[N, K]^T (C row stride ldc).  One 16 x 16 output tile
// per workgroup of 256 threads, one output per thread: the tile's 16 rows of A
// and of W are staged in LDS for a chunk of up to GF_KC k at once (each thread
// issues all its loads of the chunk before it writes any to LDS, so the chunk
// costs one memory latency), then each thread continues its float64 dot
// product over the chunk in k order.  At the fp32 models' sizes (a few hundred
// rows) this puts 6-12x more workgroups on the CUs than 64 x 64 tiles.
constexpr int GF_T = 16, GF_KC = 512, GF_PER = GF_KC / 256;
__global__ void __launch_bounds__(256) gemm_f32_kernel(const float* __restrict__ A, const float* __restrict__ W,
                                                       float* __restrict__ C, int M, int N, int K, int ldc,
                                                       int accumulate) {
  extern __shared__ float gf_lds[];
  const int m0 = blockIdx.y * GF_T, n0 = blockIdx.x * GF_T;
  const int tr = threadIdx.x / GF_T, tc = threadIdx.x % GF_T;
  double acc = 0.0;
  for (int k0 = 0; k0 < K; k0 += GF_KC) {
    const int kc = min(GF_KC, K - k0), kp = kc + 1;  // odd row pitch: the 16 W rows a k step reads hit 16 banks
    float* As = gf_lds;
    float* Ws = gf_lds + GF_T * kp;
    float ra[GF_T][GF_PER], rw[GF_T][GF_PER];
#pragma unroll
    for (int r = 0; r < GF_T; ++r)
#pragma unroll
      for (int j = 0; j < GF_PER; ++j) {
        const int k = threadIdx.x + 256 * j;
        ra[r][j] = (k < kc && m0 + r < M) ? A[(size_t)(m0 + r) * K + k0 + k] : 0.f;
        rw[r][j] = (k < kc && n0 + r < N) ? W[(size_t)(n0 + r) * K + k0 + k] : 0.f;
      }
    if (k0 > 0) __syncthreads();  // the previous chunk's reads are done
#pragma unroll
    for (int r = 0; r < GF_T; ++r)
#pragma unroll
      for (int j = 0; j < GF_PER; ++j) {
        const int k = threadIdx.x + 256 * j;
        if (k < kc) {
          As[r * kp + k] = ra[r][j];
          Ws[r * kp + k] = rw[r][j];
        }
      }
    __syncthreads();
    const float* ar = As + tr * kp;
    const float* wr = Ws + tc * kp;
#pragma unroll 16
    for (int k = 0; k < kc; ++k) acc = fma((double)ar[k], (double)wr[k], acc);
  }
  const int gm = m0 + tr, gn = n0 + tc;
  if (gm < M && gn < N) {
    float* c = C + (size_t)gm * ldc + gn;
    *c = accumulate ? (float)((double)*c + acc) : (float)acc;
  }
}

void launch_gemm_f32(const float* A, const float* W, float* C, int M, int N, int K, int ldc, bool accumulate,
                     hipStream_t s) {
  if (M == 0 || N == 0) return;
  const size_t lds = (size_t)2 * GF_T * (std::min(K, GF_KC) + 1) * sizeof(float);
  static const hipError_t attr = hipFuncSetAttribute((const void*)gemm_f32_kernel,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     (int)(2 * GF_T * (GF_KC + 1) * sizeof(float)));
  hip_check(attr, "hipFuncSetAttribute(gemm_f32)");
  hipLaunchKernelGGL(gemm_f32_kernel, dim3(ceil_div(N, GF_T), ceil_div(M, GF_T)), dim3(256), lds, s, A, W, C, M, N,
                     K, ldc, (int)accumulate);
  DLLM_LAUNCH_CHECK("gemm_f32");
}

// raw row m = b*L + l holds [q heads | k heads | v heads], each head hd wide.
__global__ void rope_split_f32_kernel(const float* __restrict__ raw, const float* __restrict__ cosb,
                                      const float* __restrict__ sinb, float* __restrict__ q, float* __restrict__ k,
                                      float* __restrict__ vt, int B, int Lq, int L, int pos0, int Hq, int Hkv,
                                      int hd) {
  const int half = hd / 2;
  const int H = Hq + 2 * Hkv;
  const long total = (long)B * Lq * H * half;
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int j = (int)(i % half);
  const int head = (int)((i / half) % H);
  const long m = i / ((long)half * H);
  const int b = (int)(m / Lq), l = (int)(m % Lq), pos = pos0 + l;
  const float* src = raw + m * (long)H * hd + (long)head * hd;
  const float x1 = src[j], x2 = src[j + half];
  if (head < Hq + Hkv) {
    const float c = cosb[(size_t)pos * half + j], sn = sinb[(size_t)pos * half + j];
    const float y1 = x1 * c - x2 * sn;
    const float y2 = x2 * c + x1 * sn;
    float* dst = head < Hq ? q + (((size_t)b * Hq + head) * Lq + l) * hd
                           : k + (((size_t)b * Hkv + (head - Hq)) * L + pos) * hd;
    dst[j] = y1;
    dst[j + half] = y2;
  } else {
    const int hv = head - Hq - Hkv;
    float* dst = vt + ((size_t)b * Hkv + hv) * hd * L;
    dst[(size_t)j * L + pos] = x1;
    dst[(size_t)(j + half) * L + pos] = x2;
  }
}

void launch_rope_split_f32(const float* raw, const float* cosb, const float* sinb, float* q, float* k, float* vt,
                           int B, int Lq, int L, int pos0, int Hq, int Hkv, int hd, hipStream_t s) {
  const long total = (long)B * Lq * (Hq + 2 * Hkv) * (hd / 2);
  if (total == 0) return;
  if (pos0 < 0 || pos0 + Lq > L) throw HipError("rope_split_f32: rows outside the sequence");
  hipLaunchKernelGGL(rope_split_f32_kernel, dim3(ceil_div(total, 256)), dim3(256), 0, s, raw, cosb, sinb, q, k, vt,
                     B, Lq, L, pos0, Hq, Hkv, hd);
  DLLM_LAUNCH_CHECK("rope_split_f32");
}

__global__ void swiglu_f32_kernel(const float* __restrict__ gate, const float* __restrict__ up,
                                  float* __restrict__ out, long n) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float g = gate[i];
  out[i] = g / (1.0f + expf(-g)) * up[i];
}

void launch_swiglu_f32(const float* gate, const float* up, float* out, long n, hipStream_t s) {
  if (n == 0) return;
  hipLaunchKernelGGL(swiglu_f32_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, s, gate, up, out, n);
  DLLM_LAUNCH_CHECK("swiglu_f32");
}

// Fixed-order block reductions over 128 threads.
__device__ double block_max128(double v, double* red) {
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const double r = fmax(red[0], red[1]);
  __syncthreads();
  return r;
}
__device__ double block_sum128(double v, double* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const double r = red[0] + red[1];
  __syncthreads();
  return r;
}

// One 128-thread block per (query, query head, sequence).  Scores for every
// key are kept in LDS (dynamic, L doubles).
__global__ void __launch_bounds__(128) attn_f32_kernel(const float* __restrict__ q, const float* __restrict__ k,
                                                       const float* __restrict__ vt, float* __restrict__ out, int Lq,
                                                       int L, int Hq, int Hkv, int hd, double scale) {
  extern __shared__ double smem[];
  double* qs = smem;          // [hd]
  double* sc = smem + 128;    // [L]
  __shared__ double red[2];
  const int l = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int kvh = h / (Hq / Hkv);
  const float* qrow = q + (((size_t)b * Hq + h) * Lq + l) * hd;
  const float* kh = k + ((size_t)b * Hkv + kvh) * L * hd;
  const float* vh = vt + ((size_t)b * Hkv + kvh) * hd * L;
  for (int d = threadIdx.x; d < hd; d += 128) qs[d] = qrow[d];
  __syncthreads();
  double mx = -INFINITY;
  for (int j = threadIdx.x; j < L; j += 128) {
    const float* kr = kh + (size_t)j * hd;
    double s = 0.0;
    for (int d = 0; d < hd; ++d) s = fma(qs[d], (double)kr[d], s);
    s *= scale;
    sc[j] = s;
    mx = fmax(mx, s);
  }
  mx = block_max128(mx, red);
  double sum = 0.0;
  for (int j = threadIdx.x; j < L; j += 128) {
    const double p = exp(sc[j] - mx);
    sc[j] = p;
    sum += p;
  }
  sum = block_sum128(sum, red);
  for (int d = threadIdx.x; d < hd; d += 128) {
    const float* vr = vh + (size_t)d * L;
    double o = 0.0;
    for (int j = 0; j < L; ++j) o = fma(sc[j], (double)vr[j], o);
    out[((size_t)b * Lq + l) * Hq * hd + (size_t)h * hd + d] = (float)(o / sum);
  }
}

void launch_attn_f32(const float* q, const float* k, const float* vt, float* out, int B, int Lq, int L, int Hq,
                     int Hkv, int hd, hipStream_t s) {
  if (B * Lq == 0) return;
  const size_t lds = (128 + (size_t)L) * sizeof(double);
  hipLaunchKernelGGL(attn_f32_kernel, dim3(Lq, Hq, B), dim3(128), lds, s, q, k, vt, out, Lq, L, Hq, Hkv, hd,
                     1.0 / sqrt((double)hd));
  DLLM_LAUNCH_CHECK("attn_f32");
}

// One 256-thread block per row.  Thread t scans v = t, t+256, ... so its first
// maximum is its lowest index; the cross-thread merge prefers the larger value,
// then the lower index.
__global__ void __launch_bounds__(256) vocab_reduce_f32_kernel(const float* __restrict__ logits, int V, int mask_id,
                                                               float* __restrict__ conf, int32_t* __restrict__ arg) {
  const int r = blockIdx.x;
  const float* row = logits + (size_t)r * V;
  float m = -INFINITY;
  int idx = 0x7fffffff;
  for (int v = threadIdx.x; v < V; v += 256) {
    if (v == mask_id) continue;
    const float x = row[v];
    if (x > m) { m = x; idx = v; }
  }
  __shared__ float sm[256];
  __shared__ int si[256];
  sm[threadIdx.x] = m;
  si[threadIdx.x] = idx;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) {
      const float m2 = sm[threadIdx.x + w];
      const int i2 = si[threadIdx.x + w];
      if (m2 > sm[threadIdx.x] || (m2 == sm[threadIdx.x] && i2 < si[threadIdx.x])) {
        sm[threadIdx.x] = m2;
        si[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  const float M = sm[0];
  const int I = si[0];
  __syncthreads();
  __shared__ double sd[256];
  double s = 0.0;
  for (int v = threadIdx.x; v < V; v += 256)
    if (v != mask_id) s += exp((double)row[v] - (double)M);
  sd[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) sd[threadIdx.x] += sd[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    conf[r] = (float)(1.0 / sd[0]);
    arg[r] = I;
  }
}

void launch_vocab_reduce_f32(const float* logits, int R, int V, int mask_id, float* conf, int32_t* argmax,
                             hipStream_t s) {
  if (R == 0) return;
  hipLaunchKernelGGL(vocab_reduce_f32_kernel, dim3(R), dim3(256), 0, s, logits, V, mask_id, conf, argmax);
  DLLM_LAUNCH_CHECK("vocab_reduce_f32");
}

}  // namespace dllm
