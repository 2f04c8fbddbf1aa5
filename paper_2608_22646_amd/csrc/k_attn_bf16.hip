// Non-causal multi-head attention with grouped KV heads, bf16 operands on
// CDNA4 matrix cores, float32 online softmax.
//
//   out[b, l, h*128 + j] = sum_k softmax_k(q[b,h,l,:] . k[b,g(h),k,:] / sqrt(128)) v[b,g(h),k,j]
//
// Every query attends to every key (no mask); g(h) = h / (Hq / Hkv).
// Workgroup = 4 wavefronts = 128 queries of one (sequence, head); wave w owns
// 32 queries.  Keys stream through LDS in tiles of 64 (K [64][128] and
// V^T [128][64], double buffered).  Per tile a wave computes
//   S^T (64 keys x 32 queries) = K . Q^T      (16 MFMAs, Q held in registers)
// so that each lane holds scores of a single query: the row max needs one
// cross-lane exchange (lane ^ 32) and the rescale factor is per lane.  Then
//   O^T (128 x 32) += V^T . P^T               (16 MFMAs)
// in IEEE half: P in [0, 1] rounded to half (11-bit significand, 8x finer than
// bf16) and V^T holding the bf16 values of v, which half represents exactly in
// its range.  The K rows of the S^T product are fed in a permuted order inside
// each 16-key group (kperm), so the scores a lane holds for one P.V slice are
// 8 consecutive keys and its V^T operand is a single 16-byte LDS read.
#include <algorithm>
#include <type_traits>

#include "kernels.h"

namespace dllm {

namespace {

constexpr int HD = 128, KT = 64, QW = 32, NW = 4;

// 2^x by the hardware instruction alone (v_exp_f32), without libm's rescaling
// for results below 2^-126: every argument here is a score minus a running
// maximum (so <= 8) whose result feeds a probability held in IEEE half or a
// sum that is at least 1, where values below 2^-126 are zero anyway.  exp2f
// spends five more VALU instructions per element on that rescaling.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// (query block, head, sequence) of this workgroup in a 1-D grid of
// nqb x Hq x B workgroups.  Workgroup i runs on XCD i % 8; each XCD takes a
// contiguous run of the (sequence, head, query block) order, so the query
// blocks of one head, which all read that head's keys and values, share one
// XCD's L2 (in grid order they were spread over all eight).
__device__ __forceinline__ int3 attn_block(int nqb, int Hq) {
  const int T = (int)gridDim.x, per = T >> 3, rem = T & 7;
  const int i = (int)blockIdx.x, x = i & 7;
  const int lin = x * per + min(x, rem) + (i >> 3);
  const int qb = lin % nqb, r = lin / nqb;
  return make_int3(qb, r % Hq, r / Hq);
}
constexpr int K_BYTES = KT * HD * 2, V_BYTES = HD * KT * 2, STAGE = K_BYTES + V_BYTES;

// XOR swizzles sized for the 64 banks (256 bytes) that one 16-lane pass of
// ds_read_b128 covers: sixteen consecutive K rows (256 B each) put a given
// chunk in sixteen different slots; sixteen consecutive V^T rows (128 B, two
// per bank line) put it in eight slots of each line parity.
__device__ __forceinline__ int k_off(int key, int chunk) {  // rows of 256 B, 16 chunks
  return key * 256 + ((chunk ^ (key & 15)) << 4);
}
__device__ __forceinline__ int v_off(int d, int chunk) {  // rows of 128 B, 8 chunks
  return K_BYTES + d * 128 + ((chunk ^ ((d >> 1) & 7)) << 4);
}
// Key order of the S^T MFMA rows inside each 16-key group: row i takes key
// kperm(i) (bits 2 and 3 swapped).  A lane's scores then come out as 8
// consecutive keys per P.V slice (register 4b + c of lane half h holds key
// 8h + 4b + c of the group), so its V^T operand is one 16-byte chunk -- one
// conflict-free ds_read_b128 instead of two 8-byte reads that two lanes of a
// pass share banks with.
__device__ __forceinline__ int kperm(int i) { return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1); }
// max / sum of x over lanes l and l ^ 32 (the two halves holding one query's
// scores): v_permlane32_swap with both operands x yields, at every lane, the
// values of the lower and the upper half at that position -- a VALU exchange
// instead of an LDS round trip (ds_bpermute)
__device__ __forceinline__ float max_pair32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_pair32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__global__ void __launch_bounds__(256, 1) attn_bf16_kernel(const bf16_t* __restrict__ q, const bf16_t* __restrict__ k,
                                                           const f16_t* __restrict__ vt, bf16_t* __restrict__ out,
                                                           int Lq, int L, int Hq, int Hkv) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int3 wb = attn_block((Lq + QW * NW - 1) / (QW * NW), Hq);
  const int h = wb.y, b = wb.z, g = h / (Hq / Hkv);
  const int q0 = wb.x * (QW * NW) + wave * QW;
  const int lq = lane & 31, half = lane >> 5;
  const bf16_t* kh = k + ((size_t)b * Hkv + g) * L * HD;
  const f16_t* vh = vt + ((size_t)b * Hkv + g) * HD * L;

  // Q as the B operand: lane holds query q0 + lq, dims 16*ks + 8*half .. +7.
  bf16x8_t qf[8];
  {
    const int qi = q0 + lq;
    const bf16_t* qrow = q + (((size_t)b * Hq + h) * Lq + (qi < Lq ? qi : 0)) * HD;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      qf[ks] = *reinterpret_cast<const bf16x8_t*>(qrow + ks * 16 + half * 8);
      if (qi >= Lq) qf[ks] = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    }
  }

  // tile loader: 4 x 16 B of K and 4 x 16 B of V^T per thread
  uint4 rk[4], rv[4];
  auto gload = [&](int t0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + 256 * i;
      const int key = e >> 4, ch = e & 15;  // K: 64 rows x 16 chunks
      const int gk = t0 + key;
      rk[i] = gk < L ? *reinterpret_cast<const uint4*>(kh + (size_t)gk * HD + ch * 8) : make_uint4(0, 0, 0, 0);
      const int d = e >> 3, vc = e & 7;     // V^T: 128 rows x 8 chunks
      const int gv = t0 + vc * 8;
      if ((L & 7) == 0 && gv + 8 <= L) {
        rv[i] = *reinterpret_cast<const uint4*>(vh + (size_t)d * L + gv);
      } else {
        uint16_t tmp[8];
        for (int x = 0; x < 8; ++x) tmp[x] = (gv + x < L) ? vh[(size_t)d * L + gv + x] : (uint16_t)0;
        rv[i] = *reinterpret_cast<uint4*>(tmp);
      }
    }
  };
  auto sstore = [&](int buf) {
    char* base = lds + buf * STAGE;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + 256 * i;
      *reinterpret_cast<uint4*>(base + k_off(e >> 4, e & 15)) = rk[i];
      *reinterpret_cast<uint4*>(base + v_off(e >> 3, e & 7)) = rv[i];
    }
  };

  f32x16_t o[4];
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[ds][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sc = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)

  const int ntiles = (L + KT - 1) / KT;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) gload((t + 1) * KT);
    const char* base = lds + buf * STAGE;

    // S^T = K . Q^T for keys 32*st + (rows), queries = lanes; the K fragments
    // are read ahead of their MFMAs
    f32x16_t s[2];
    bf16x8_t kf[2][8];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int ks = 0; ks < 8; ++ks)
        kf[st][ks] = *reinterpret_cast<const bf16x8_t*>(base + k_off(st * 32 + kperm(lq), ks * 2 + half));
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[st][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st][ks], qf[ks], s[st], 0, 0, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
    for (int x = 0; x < 8; ++x) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    // scale into the log2 domain, mask keys past L, tile max
    const int t0 = t * KT;
    float mt = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = t0 + st * 32 + kperm(8 * (r >> 2) + 4 * half + (r & 3));
        const float x = key < L ? s[st][r] * sc : -INFINITY;
        s[st][r] = x;
        mt = fmaxf(mt, x);
      }
    mt = max_pair32(mt);
    const float m_new = fmaxf(m_run, mt);
    const float alpha = exp2_hw(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2_hw(s[st][r] - m_new);
        s[st][r] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[ds][r] *= alpha;

    // O^T += V^T . P^T over four 16-key slices
#pragma unroll
    for (int jk = 0; jk < 4; ++jk) {
      f16x8_t pf;
      const int st = jk >> 1, r0 = (jk & 1) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = (_Float16)s[st][r0 + e];
      // slot e: key 16jk + 8*half + e (kperm), one 16-byte V^T chunk
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) {
        const int d = ds * 32 + lq;
        const f16x8_t vf = *reinterpret_cast<const f16x8_t*>(base + v_off(d, 2 * jk + half));
        o[ds] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pf, o[ds], 0, 0, 0);
      }
    }
    if (t + 1 < ntiles) sstore(buf ^ 1);
    __syncthreads();
  }

  const float l_tot = sum_pair32(l_run);
  const float inv = 1.0f / l_tot;
  const int qi = q0 + lq;
  if (qi >= Lq) return;
  bf16_t* orow = out + ((size_t)b * Lq + qi) * ((size_t)Hq * HD) + (size_t)h * HD;
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d = ds * 32 + 8 * rg + 4 * half;
      uint2 w;
      w.x = pack_bf16x2(o[ds][rg * 4 + 0] * inv, o[ds][rg * 4 + 1] * inv);
      w.y = pack_bf16x2(o[ds][rg * 4 + 2] * inv, o[ds][rg * 4 + 3] * inv);
      *reinterpret_cast<uint2*>(orow + d) = w;
    }
}


// ---------------------------------------------------------------------------
// Streaming variant for sequences whose length is a multiple of 8: NW
// wavefronts x 32 queries per workgroup (NW = 8: two waves per SIMD, so one
// wave's softmax overlaps the other's MFMAs, and each K/V tile serves 256
// queries).  K and V^T tiles are copied straight into a 3-stage LDS ring with
// buffer_load_dwordx4 ... lds.  Keys past L are masked; their K rows read as
// zero through the buffer bound, and their V^T columns hold either the next
// d-row's (finite) values or, past the end of the head, zeros.  The 1/sqrt(hd) * log2(e) scale is folded into the
// exp2 argument, and the running maximum is only raised when a tile's maximum
// exceeds it by more than 8 (log2 units): unnormalised probabilities then stay
// below 2^8 (exact to half's relative precision) and the O / l rescale is
// skipped for most tiles.
typedef __attribute__((address_space(3))) void* lds_ptr_t;

template <int N>
__device__ __forceinline__ void wait_vmcnt_a() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void barrier_nofence_a() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int NW>
__global__ void __launch_bounds__(64 * NW, 1) attn_stream_kernel(const bf16_t* __restrict__ q,
                                                                 const bf16_t* __restrict__ k,
                                                                 const f16_t* __restrict__ vt,
                                                                 bf16_t* __restrict__ out, int Lq, int L, int Hq, int Hkv) {
#if defined(__HIP_DEVICE_COMPILE__)
  // D tiles in flight ahead of the one in use
  constexpr int D = 2, S = D + 1, PER_STAGE = 32 / NW;  // 16 K + 16 V^T DMA instructions per tile
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int3 wb = attn_block((Lq + QW * NW - 1) / (QW * NW), Hq);
  const int h = wb.y, b = wb.z, g = h / (Hq / Hkv);
  const int q0 = wb.x * (QW * NW) + wave * QW;
  const int lq = lane & 31, half = lane >> 5;
  const bf16_t* kh = k + ((size_t)b * Hkv + g) * L * HD;
  const f16_t* vh = vt + ((size_t)b * Hkv + g) * HD * L;

  bf16x8_t qf[8];
  {
    const int qi = q0 + lq;
    const bf16_t* qrow = q + (((size_t)b * Hq + h) * Lq + (qi < Lq ? qi : 0)) * HD;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      qf[ks] = *reinterpret_cast<const bf16x8_t*>(qrow + ks * 16 + half * 8);
      if (qi >= Lq) qf[ks] = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    }
  }

  // DMA: K instruction i fills keys 4i..4i+3 (rows of 256 B, lane l -> key
  // 4i + l/16, slot l%16 holding chunk (l%16) ^ (key & 15)); V^T instruction i
  // fills d rows 8i..8i+7 (rows of 128 B, lane l -> d = 8i + l/8, slot l%8
  // holding chunk (l%8) ^ ((d >> 1) & 7)).  Wave w issues instructions w, w + NW, ...
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)kh, 0, L * HD * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)vh, 0, HD * L * 2, 0x00020000);
  constexpr int PK = 16 / NW;
  uint32_t vok[PK], vov[PK];
#pragma unroll
  for (int j = 0; j < PK; ++j) {
    const int i = wave + NW * j;
    const int key = 4 * i + (lane >> 4), kc = (lane & 15) ^ (key & 15);
    vok[j] = (uint32_t)((key * HD + kc * 8) * 2);
    const int d = 8 * i + (lane >> 3), vc = (lane & 7) ^ ((d >> 1) & 7);
    vov[j] = (uint32_t)(((size_t)d * L + vc * 8) * 2);
  }
  auto issue = [&](int t) {
    char* base = lds + (t % S) * STAGE;
    const int t0 = t * KT;
#pragma unroll
    for (int j = 0; j < PK; ++j) {
      const int i = wave + NW * j;
      // the tile offset goes in the per-lane offset, which the buffer bound
      // checks: reads past the end of this head's K or V^T return zeros
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr_t)(base + i * 1024), 16, vok[j] + t0 * HD * 2, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_ptr_t)(base + K_BYTES + i * 1024), 16, vov[j] + t0 * 2, 0, 0,
                                               0);
    }
  };

  f32x16_t o[4];
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[ds][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sc = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)

  // P (half) slot e of slice jk holds key 16 jk + 8 half + e (kperm), so a
  // lane's V^T operand of the slice is the 16-byte chunk 2 jk + half of row d
  auto to_half = [&](const f32x16_t (&p2)[2], int jk) {
    f16x8_t pf;
#pragma unroll
    for (int e = 0; e < 8; ++e) pf[e] = (_Float16)p2[jk >> 1][(jk & 1) * 8 + e];
    return pf;
  };

  const int ntiles = (L + KT - 1) / KT;
#pragma unroll
  for (int s = 0; s < D; ++s)
    if (s < ntiles) issue(s);
  for (int t = 0; t < ntiles; ++t) {
    if (t + 1 < ntiles)
      wait_vmcnt_a<PER_STAGE * (D - 1)>();
    else
      wait_vmcnt_a<0>();
    barrier_nofence_a();  // tile t visible; every wave is done with the slot refilled next
    if (t + D < ntiles) issue(t + D);
    const char* base = lds + (t % S) * STAGE;

    // S^T: all 16 K fragments are read before the MFMAs that use them, the
    // second 32-key half's reads under the first half's MFMAs (read one,
    // multiply one, each read waiting for its LDS round trip, runs ~2x slower)
    f32x16_t s2[2];
    bf16x8_t kf[8][2];
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
#pragma unroll
      for (int st = 0; st < 2; ++st)
        kf[ks][st] = *reinterpret_cast<const bf16x8_t*>(base + k_off(st * 32 + kperm(lq), ks * 2 + half));
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r) s2[st][r] = 0.f;
    // the two 32-key halves' accumulation chains alternate
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
#pragma unroll
      for (int st = 0; st < 2; ++st) s2[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks][st], qf[ks], s2[st], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);  // K reads run six ahead of their MFMAs
    for (int x = 0; x < 10; ++x) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
    const int t0 = t * KT;
    float mt = -INFINITY;
    if (t0 + KT <= L) {
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s2[st][r]);
    } else {
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = t0 + st * 32 + kperm(8 * (r >> 2) + 4 * half + (r & 3));
          if (key >= L) s2[st][r] = -INFINITY;
          mt = fmaxf(mt, s2[st][r]);
        }
    }
    mt = max_pair32(mt) * sc;
    // raise the running maximum only when it grows by more than 2^8
    if (__ballot(mt > m_run + 8.0f) != 0ull) {
      const float m_new = fmaxf(m_run, mt);
      const float alpha = exp2_hw(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[ds][r] *= alpha;
    }
    float psum = 0.f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2_hw(fmaf(s2[st][r], sc, -m_run));
        s2[st][r] = p;
        psum += p;
      }
    l_run += psum;
    // O^T += V^T P^T: each slice's four V^T reads are issued under the
    // previous slice's MFMAs
    f16x8_t vf[2][4];
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) vf[0][ds] = *reinterpret_cast<const f16x8_t*>(base + v_off(ds * 32 + lq, half));
#pragma unroll
    for (int jk = 0; jk < 4; ++jk) {
      if (jk < 3) {
#pragma unroll
        for (int ds = 0; ds < 4; ++ds)
          vf[(jk + 1) & 1][ds] = *reinterpret_cast<const f16x8_t*>(base + v_off(ds * 32 + lq, 2 * (jk + 1) + half));
      }
      const f16x8_t pf = to_half(s2, jk);
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) o[ds] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf[jk & 1][ds], pf, o[ds], 0, 0, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // slice 0's V^T reads
    for (int x = 0; x < 12; ++x) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one V^T read of the next slice
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  }

  const float l_tot = sum_pair32(l_run);
  const float inv = 1.0f / l_tot;
  const int qi = q0 + lq;
  if (qi >= Lq) return;
  bf16_t* orow = out + ((size_t)b * Lq + qi) * ((size_t)Hq * HD) + (size_t)h * HD;
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d = ds * 32 + 8 * rg + 4 * half;
      uint2 w;
      w.x = pack_bf16x2(o[ds][rg * 4 + 0] * inv, o[ds][rg * 4 + 1] * inv);
      w.y = pack_bf16x2(o[ds][rg * 4 + 2] * inv, o[ds][rg * 4 + 3] * inv);
      *reinterpret_cast<uint2*>(orow + d) = w;
    }
#endif
}


// Key-split variant with 32-key tiles for short launches (batch 1 at a few
// hundred tokens): a workgroup owns 32 QG queries of one (sequence, head) and
// runs QG x 4 waves -- wave w takes queries 32 (w % QG) .. +31 and the key
// tiles 4u + w / QG, u = 0, 1, ... -- so the grid reaches every CU and each
// wave's chain of dependent tiles is a quarter of the sequence.  A step brings
// four 32-key tiles (K [32][128], V^T [128][32], 16 KiB each) into a 2-stage
// LDS ring by LDS-DMA; at the end the four key groups' running (max, sum,
// output) states are merged in group order through LDS.
constexpr int KT2 = 32, KB2 = KT2 * HD * 2, TB2 = 2 * KB2, KGRP = 4, STEP2 = KGRP * TB2;

__device__ __forceinline__ int v2_off(int d, int chunk) {  // V^T rows of 64 B, 4 chunks
  return KB2 + d * 64 + ((chunk ^ ((d >> 2) & 3)) << 4);
}

template <int QG>
__global__ void __launch_bounds__(64 * QG * KGRP, 1) attn_kv4_kernel(const bf16_t* __restrict__ q,
                                                                    const bf16_t* __restrict__ k,
                                                                    const f16_t* __restrict__ vt,
                                                                    bf16_t* __restrict__ out, int Lq, int L, int Hq, int Hkv) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int NW = QG * KGRP, S = 2;
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qg = wave % QG, kg = wave / QG;
  const int3 wb = attn_block((Lq + QW * QG - 1) / (QW * QG), Hq);
  const int h = wb.y, b = wb.z, g = h / (Hq / Hkv);
  const int q0 = wb.x * (QW * QG) + qg * QW;
  const int lq = lane & 31, half = lane >> 5;
  const bf16_t* kh = k + ((size_t)b * Hkv + g) * L * HD;
  const f16_t* vh = vt + ((size_t)b * Hkv + g) * HD * L;

  // DMA of a step: 64 instructions of 1 KiB, instruction j (tile j / 16,
  // part j % 16) issued by wave j % NW.  K part i < 8: keys 4i + l/16, slot
  // l%16 holding chunk (l%16) ^ (key & 15); V^T part i >= 8: d rows
  // 16 (i - 8) + l/4, slot l%4 holding chunk (l%4) ^ ((d >> 2) & 3).  Reads
  // past the end of this head's K or V^T return zeros (buffer bound).
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)kh, 0, L * HD * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)vh, 0, HD * L * 2, 0x00020000);
  constexpr int PJ = (64 + NW - 1) / NW;
  uint32_t voff[PJ];
#pragma unroll
  for (int x = 0; x < PJ; ++x) {
    const int j = wave + NW * x, part = j & 15;
    if (part < 8) {
      const int key = 4 * part + (lane >> 4), kc = (lane & 15) ^ (key & 15);
      voff[x] = (uint32_t)((key * HD + kc * 8) * 2);
    } else {
      const int d = 16 * (part - 8) + (lane >> 2), vc = (lane & 3) ^ ((d >> 2) & 3);
      voff[x] = (uint32_t)(((size_t)d * L + vc * 8) * 2);
    }
  }
  auto issue = [&](int u) {
    char* base = lds + (u % S) * STEP2;
#pragma unroll
    for (int x = 0; x < PJ; ++x) {
      const int j = wave + NW * x;
      if (j < 64) {
        const int tile = j >> 4, part = j & 15, t0 = (KGRP * u + tile) * KT2;
        char* dst = base + tile * TB2 + part * 1024;
        if (part < 8)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr_t)dst, 16, voff[x] + t0 * HD * 2, 0, 0, 0);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_ptr_t)dst, 16, voff[x] + t0 * 2, 0, 0, 0);
      }
    }
  };

  const int nsteps = (L + KGRP * KT2 - 1) / (KGRP * KT2);
  issue(0);

  bf16x8_t qf[8];
  {
    const int qi = q0 + lq;
    const bf16_t* qrow = q + (((size_t)b * Hq + h) * Lq + (qi < Lq ? qi : 0)) * HD;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      qf[ks] = *reinterpret_cast<const bf16x8_t*>(qrow + ks * 16 + half * 8);
      if (qi >= Lq) qf[ks] = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    }
  }

  f32x16_t o[4];
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[ds][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sc = 1.4426950408889634f / sqrtf((float)HD);

  for (int u = 0; u < nsteps; ++u) {
    wait_vmcnt_a<0>();
    barrier_nofence_a();  // step u visible; slot (u + 1) % 2 free
    if (u + 1 < nsteps) issue(u + 1);
    const int t0 = (KGRP * u + kg) * KT2;
    if (t0 >= L) continue;  // this group has no keys left in the last step
    const char* base = lds + (u % S) * STEP2 + kg * TB2;

    // two independent accumulation chains (even and odd 16-dim slices); the K
    // fragments are read in batches of KPF ahead of the MFMAs that use them
    // (two at three waves per SIMD, where eight would not fit the registers)
    constexpr int KPF = QG == 3 ? 2 : 8;
    f32x16_t s2, s2b;
#pragma unroll
    for (int r = 0; r < 16; ++r) s2[r] = s2b[r] = 0.f;
#pragma unroll
    for (int k0 = 0; k0 < 8; k0 += KPF) {
      bf16x8_t kf[KPF];
#pragma unroll
      for (int i = 0; i < KPF; ++i)
        kf[i] = *reinterpret_cast<const bf16x8_t*>(base + k_off(kperm(lq), (k0 + i) * 2 + half));
#pragma unroll
      for (int i = 0; i < KPF; i += 2) {
        s2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i], qf[k0 + i], s2, 0, 0, 0);
        s2b = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i + 1], qf[k0 + i + 1], s2b, 0, 0, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x100, KPF, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, KPF, 0);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) s2[r] += s2b[r];
    float mt = -INFINITY;
    if (t0 + KT2 <= L) {
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s2[r]);
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = t0 + kperm(8 * (r >> 2) + 4 * half + (r & 3));
        if (key >= L) s2[r] = -INFINITY;
        mt = fmaxf(mt, s2[r]);
      }
    }
    mt = max_pair32(mt) * sc;
    if (__ballot(mt > m_run + 8.0f) != 0ull) {
      const float m_new = fmaxf(m_run, mt);
      const float alpha = exp2_hw(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[ds][r] *= alpha;
    }
    float psum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = exp2_hw(fmaf(s2[r], sc, -m_run));
      s2[r] = p;
      psum += p;
    }
    l_run += psum;

    // slot e of slice jk: key 16jk + 8*half + e (kperm), one 16-byte V^T
    // chunk; a slice's four V^T fragments are read before its MFMAs (left to
    // the compiler at three waves per SIMD, short of registers)
#pragma unroll
    for (int jk = 0; jk < 2; ++jk) {
      f16x8_t vf[4];
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
        vf[ds] = *reinterpret_cast<const f16x8_t*>(base + v2_off(ds * 32 + lq, 2 * jk + half));
      f16x8_t pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = (_Float16)s2[jk * 8 + e];
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) o[ds] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf[ds], pf, o[ds], 0, 0, 0);
      if (QG < 3) {
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      }
    }
  }

  // merge the four key groups of each query group in group order (the ring
  // is idle once every wave has passed the barrier)
  __syncthreads();
  if (QG <= 2) {
    // every wave leaves its 64 floats of o as 16 lane-contiguous float4 rows,
    // then (m, l); wave (qg, kg) then finishes output dimensions 32 kg .. of
    // query group qg (the same operations, in the same order, as a merge by
    // one wave per query group), stages them as bf16 rows and the workgroup
    // stores whole 256-byte rows
    constexpr int SLOT = 17 * 64;                       // float4s per wave
    constexpr int OPK = 272;                            // staged row pitch (bytes)
    char* stg = lds + (size_t)NW * SLOT * 16;           // [QG * 32][OPK]
    float4* xo = reinterpret_cast<float4*>(lds) + (size_t)wave * SLOT + lane;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq)
        xo[(ds * 4 + rq) * 64] = make_float4(o[ds][4 * rq], o[ds][4 * rq + 1], o[ds][4 * rq + 2], o[ds][4 * rq + 3]);
    xo[16 * 64] = make_float4(m_run, l_run, 0.f, 0.f);
    __syncthreads();
    const float4* x4 = reinterpret_cast<const float4*>(lds) + lane;
    float me[KGRP], le[KGRP], m = -INFINITY;
#pragma unroll
    for (int e = 0; e < KGRP; ++e) {
      const float4 ml = x4[(size_t)(qg + QG * e) * SLOT + 16 * 64];
      me[e] = ml.x;
      le[e] = ml.y;
      m = fmaxf(m, ml.x);
    }
    float acc[16], l_lane = 0.f;
#pragma unroll
    for (int e = 0; e < KGRP; ++e) {
      // a group that saw no key (m = -inf) contributes nothing
      const float ae = me[e] == -INFINITY ? 0.f : exp2_hw(me[e] - m);
      const float4* xe = x4 + (size_t)(qg + QG * e) * SLOT + kg * 4 * 64;
      l_lane = e == 0 ? le[e] * ae : fmaf(le[e], ae, l_lane);
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const float4 v = xe[rq * 64];
        if (e == 0) {
          acc[4 * rq] = v.x * ae;
          acc[4 * rq + 1] = v.y * ae;
          acc[4 * rq + 2] = v.z * ae;
          acc[4 * rq + 3] = v.w * ae;
        } else {
          acc[4 * rq] += v.x * ae;
          acc[4 * rq + 1] += v.y * ae;
          acc[4 * rq + 2] += v.z * ae;
          acc[4 * rq + 3] += v.w * ae;
        }
      }
    }
    const float inv = 1.0f / sum_pair32(l_lane);
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d = kg * 32 + 8 * rg + 4 * half;
      uint2 w;
      w.x = pack_bf16x2(acc[rg * 4 + 0] * inv, acc[rg * 4 + 1] * inv);
      w.y = pack_bf16x2(acc[rg * 4 + 2] * inv, acc[rg * 4 + 3] * inv);
      *reinterpret_cast<uint2*>(stg + (qg * QW + lq) * OPK + d * 2) = w;
    }
    __syncthreads();
    const int qb0 = wb.x * (QW * QG);
    for (int it = tid; it < QG * QW * 16; it += NW * 64) {
      const int row = it >> 4, ch = it & 15, qi = qb0 + row;
      if (qi < Lq)
        *reinterpret_cast<uint4*>(out + ((size_t)b * Lq + qi) * ((size_t)Hq * HD) + (size_t)h * HD + ch * 8) =
            *reinterpret_cast<const uint4*>(stg + row * OPK + ch * 16);
    }
    return;
  }
  // three query groups: groups 1..3 leave their 64 floats of o as 16
  // lane-contiguous float4 rows, then (m, l), for group 0 to merge
  constexpr int XW = 17 * 64 * 4;  // floats per handed-over wave
  if (kg > 0) {
    float4* xo = reinterpret_cast<float4*>(lds) + (size_t)(wave - QG) * (XW / 4) + lane;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq)
        xo[(ds * 4 + rq) * 64] = make_float4(o[ds][4 * rq], o[ds][4 * rq + 1], o[ds][4 * rq + 2], o[ds][4 * rq + 3]);
    xo[16 * 64] = make_float4(m_run, l_run, 0.f, 0.f);
  }
  __syncthreads();
  if (kg > 0) return;
  {
    const float4* x4 = reinterpret_cast<const float4*>(lds) + lane;
    float me[KGRP - 1], le[KGRP - 1];
    float m = m_run;
#pragma unroll
    for (int e = 1; e < KGRP; ++e) {
      const float4 ml = x4[(size_t)(qg + QG * (e - 1)) * (XW / 4) + 16 * 64];
      me[e - 1] = ml.x;
      le[e - 1] = ml.y;
      m = fmaxf(m, ml.x);
    }
    // a group that saw no key (m = -inf) contributes nothing
    const float a0 = m_run == -INFINITY ? 0.f : exp2_hw(m_run - m);
    l_run *= a0;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[ds][r] *= a0;
#pragma unroll
    for (int e = 1; e < KGRP; ++e) {
      const float4* xe = x4 + (size_t)(qg + QG * (e - 1)) * (XW / 4);
      const float ae = me[e - 1] == -INFINITY ? 0.f : exp2_hw(me[e - 1] - m);
      l_run += le[e - 1] * ae;
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const float4 v = xe[(ds * 4 + rq) * 64];
          o[ds][4 * rq] += v.x * ae;
          o[ds][4 * rq + 1] += v.y * ae;
          o[ds][4 * rq + 2] += v.z * ae;
          o[ds][4 * rq + 3] += v.w * ae;
        }
    }
  }

  // normalise and stage the wave's 32 output rows (bf16, 272-byte pitch) in
  // the hand-over slot of its group-1 partner, which only this wave reads,
  // then store them as whole 256-byte rows
  const float l_tot = sum_pair32(l_run);
  const float inv = 1.0f / l_tot;
  constexpr int OP = 272;
  char* stg = lds + (size_t)qg * XW * 4;
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d = ds * 32 + 8 * rg + 4 * half;
      uint2 w;
      w.x = pack_bf16x2(o[ds][rg * 4 + 0] * inv, o[ds][rg * 4 + 1] * inv);
      w.y = pack_bf16x2(o[ds][rg * 4 + 2] * inv, o[ds][rg * 4 + 3] * inv);
      *reinterpret_cast<uint2*>(stg + lq * OP + d * 2) = w;
    }
  __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0): this wave's writes landed
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int row = it * 4 + (lane >> 4), ch = lane & 15, qi = q0 + row;
    if (qi < Lq)
      *reinterpret_cast<uint4*>(out + ((size_t)b * Lq + qi) * ((size_t)Hq * HD) + (size_t)h * HD + ch * 8) =
          *reinterpret_cast<const uint4*>(stg + row * OP + ch * 16);
  }
#endif
}

// Key-split variant for at most 32 queries per (sequence, head) -- a cached
// step's block rows against every cached position: the keys of a head are
// split over NS workgroups of NWS waves, wave w of split s taking the 32-key
// tiles s nt / NS + w, + NWS, ... (nt tiles in all).  With one query group a
// tile is read by exactly one wave, so its K and V^T fragments go straight
// from memory into registers (the next tile's loads in flight under the
// current one's MFMAs): no LDS ring and no barrier in the loop.  The waves'
// running (max, sum, output) states are merged in wave order through LDS; with
// NS > 1 the workgroup publishes the merged state (device-coherent stores) and
// takes a ticket of its (sequence, head), and the last of the NS workgroups
// merges the NS states in split order (wave w the output dimensions 32 w ..),
// writes the bf16 rows and re-arms the ticket.  Tickets start at zero (the
// forward's embedding kernel clears them) and every launch leaves them zero.
constexpr int CPOL_SC1_A = 16;  // cache-policy bit: coherent at device (agent) scope
constexpr int SPLIT_STATE = 17 * 64 * 16;  // bytes of one published state: 16 float4 of o + (m, l) per lane

template <int NWS>
__global__ void __launch_bounds__(64 * NWS, 1) attn_split_kernel(const bf16_t* __restrict__ q,
                                                                 const bf16_t* __restrict__ k,
                                                                 const f16_t* __restrict__ vt,
                                                                 bf16_t* __restrict__ out, float* __restrict__ part,
                                                                 int* __restrict__ ticket, int Lq, int L, int Hq,
                                                                 int Hkv, int NS) {
#if defined(__HIP_DEVICE_COMPILE__)
  __shared__ float4 xch[NWS > 1 ? NWS - 1 : 1][17][64];
  __shared__ int last_flag;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // XCD-aware 1-D grid over (sequence, head, split), the splits of a head adjacent
  const int T = (int)gridDim.x, per = T >> 3, rem = T & 7, xi = (int)blockIdx.x & 7;
  const int lin = xi * per + min(xi, rem) + ((int)blockIdx.x >> 3);
  const int s = lin % NS, bh = lin / NS, h = bh % Hq, b = bh / Hq, g = h / (Hq / Hkv);
  const int lq = lane & 31, half = lane >> 5;
  const int nt = (L + KT2 - 1) / KT2, tb = (int)((long)s * nt / NS), te = (int)((long)(s + 1) * nt / NS);
  const bf16_t* kh = k + ((size_t)b * Hkv + g) * L * HD;
  const f16_t* vh = vt + ((size_t)b * Hkv + g) * HD * L;
  // reads past this head's K or V^T return zeros (buffer bound)
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)kh, 0, L * HD * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)vh, 0, HD * L * 2, 0x00020000);
  typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
  // K operand i of a tile at key t0: key t0 + kperm(lq), dimensions 16 i + 8 half ..;
  // V^T operand (jk, ds): dimension 32 ds + lq, keys t0 + 16 jk + 8 half ..
  const uint32_t ko = (uint32_t)((kperm(lq) * HD + half * 8) * 2), vo = (uint32_t)((lq * L + half * 8) * 2);
  u32x4_t kb[2][8], vb[2][8];
  auto load = [&](int t, int set) {
    const int t0 = t * KT2;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      kb[set][i] = __builtin_amdgcn_raw_buffer_load_b128(rk, ko + (uint32_t)((t0 * HD + 16 * i) * 2), 0, 0);
#pragma unroll
    for (int jk = 0; jk < 2; ++jk)
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
        vb[set][jk * 4 + ds] =
            __builtin_amdgcn_raw_buffer_load_b128(rv, vo + (uint32_t)((ds * 32 * L + t0 + 16 * jk) * 2), 0, 0);
  };

  bf16x8_t qf[8];
  {
    const int qi = lq;
    const bf16_t* qrow = q + (((size_t)b * Hq + h) * Lq + (qi < Lq ? qi : 0)) * HD;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      qf[ks] = *reinterpret_cast<const bf16x8_t*>(qrow + ks * 16 + half * 8);
      if (qi >= Lq) qf[ks] = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    }
  }
  f32x16_t o[4];
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[ds][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sc = 1.4426950408889634f / sqrtf((float)HD);

  // one 32-key tile from fragment set S_ (compile-time), the next tile's
  // fragments loading into the other set meanwhile
  auto step = [&](int t, auto set_c) {
    constexpr int cur = decltype(set_c)::value;
    if (t + NWS < te) load(t + NWS, cur ^ 1);
    const int t0 = t * KT2;
    f32x16_t s2, s2b;
#pragma unroll
    for (int r = 0; r < 16; ++r) s2[r] = s2b[r] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      s2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kb[cur][i]), qf[i], s2, 0, 0, 0);
      s2b = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kb[cur][i + 1]), qf[i + 1], s2b, 0,
                                                    0, 0);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) s2[r] += s2b[r];
    float mt = -INFINITY;
    if (t0 + KT2 <= L) {
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s2[r]);
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = t0 + kperm(8 * (r >> 2) + 4 * half + (r & 3));
        if (key >= L) s2[r] = -INFINITY;
        mt = fmaxf(mt, s2[r]);
      }
    }
    mt = max_pair32(mt) * sc;
    if (__ballot(mt > m_run + 8.0f) != 0ull) {
      const float m_new = fmaxf(m_run, mt);
      const float alpha = exp2_hw(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[ds][r] *= alpha;
    }
    float psum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = exp2_hw(fmaf(s2[r], sc, -m_run));
      s2[r] = p;
      psum += p;
    }
    l_run += psum;
#pragma unroll
    for (int jk = 0; jk < 2; ++jk) {
      f16x8_t pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = (_Float16)s2[jk * 8 + e];
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
        o[ds] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, vb[cur][jk * 4 + ds]), pf, o[ds],
                                                       0, 0, 0);
    }
  };
  int t = tb + wave;
  if (t < te) load(t, 0);
  while (t < te) {
    step(t, std::integral_constant<int, 0>{});
    t += NWS;
    if (t >= te) break;
    step(t, std::integral_constant<int, 1>{});
    t += NWS;
  }

  // merge the waves in wave order; a wave that saw no key (m = -inf) adds nothing
  if (NWS > 1) {
    if (wave > 0) {
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq)
          xch[wave - 1][ds * 4 + rq][lane] =
              make_float4(o[ds][4 * rq], o[ds][4 * rq + 1], o[ds][4 * rq + 2], o[ds][4 * rq + 3]);
      xch[wave - 1][16][lane] = make_float4(m_run, l_run, 0.f, 0.f);
    }
    __syncthreads();
    if (wave == 0) {
      float m = m_run;
#pragma unroll
      for (int e = 0; e < NWS - 1; ++e) m = fmaxf(m, xch[e][16][lane].x);
      const float a0 = m_run == -INFINITY ? 0.f : exp2_hw(m_run - m);
      l_run *= a0;
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[ds][r] *= a0;
#pragma unroll
      for (int e = 0; e < NWS - 1; ++e) {
        const float me = xch[e][16][lane].x, le = xch[e][16][lane].y;
        const float ae = me == -INFINITY ? 0.f : exp2_hw(me - m);
        l_run += le * ae;
#pragma unroll
        for (int ds = 0; ds < 4; ++ds)
#pragma unroll
          for (int rq = 0; rq < 4; ++rq) {
            const float4 v = xch[e][ds * 4 + rq][lane];
            o[ds][4 * rq] += v.x * ae;
            o[ds][4 * rq + 1] += v.y * ae;
            o[ds][4 * rq + 2] += v.z * ae;
            o[ds][4 * rq + 3] += v.w * ae;
          }
      }
      m_run = m;
    }
  }

  auto store_rows = [&](const f32x16_t* oo, int ds0, int nds, float l) {
    const float inv = 1.0f / sum_pair32(l);
    if (lq >= Lq) return;
    bf16_t* orow = out + ((size_t)b * Lq + lq) * ((size_t)Hq * HD) + (size_t)h * HD;
    for (int ds = ds0; ds < ds0 + nds; ++ds)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int d = ds * 32 + 8 * rg + 4 * half;
        uint2 w;
        w.x = pack_bf16x2(oo[ds - ds0][rg * 4 + 0] * inv, oo[ds - ds0][rg * 4 + 1] * inv);
        w.y = pack_bf16x2(oo[ds - ds0][rg * 4 + 2] * inv, oo[ds - ds0][rg * 4 + 3] * inv);
        *reinterpret_cast<uint2*>(orow + d) = w;
      }
  };
  if (NS == 1) {
    if (wave == 0) store_rows(o, 0, 4, l_run);
    return;
  }

  // publish the workgroup's state: lane-contiguous float4s [17][64] per (sequence, head, split)
  const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc((void*)part, 0, 0x7fffffff, 0x00020000);
  if (wave == 0) {
    const uint32_t base = (uint32_t)(((size_t)bh * NS + s) * SPLIT_STATE) + lane * 16;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const u32x4_t v = {__float_as_uint(o[ds][4 * rq]), __float_as_uint(o[ds][4 * rq + 1]),
                           __float_as_uint(o[ds][4 * rq + 2]), __float_as_uint(o[ds][4 * rq + 3])};
        __builtin_amdgcn_raw_buffer_store_b128(v, rp, base + (ds * 4 + rq) * 1024, 0, CPOL_SC1_A);
      }
    const u32x4_t ml = {__float_as_uint(m_run), __float_as_uint(l_run), 0u, 0u};
    __builtin_amdgcn_raw_buffer_store_b128(ml, rp, base + 16 * 1024, 0, CPOL_SC1_A);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) last_flag = atomicAdd(ticket + bh, 1) == NS - 1;
  __syncthreads();
  if (!last_flag) return;

  // last workgroup of the head: wave w merges output dimensions 32 ds .. 32 ds
  // + 31, ds = w, w + NWS, .., of every split in split order (the merged m first)
  for (int ds = wave; ds < 4; ds += NWS) {
    // the splits' states in rounds of ZB, all loads of a round in flight at
    // once; an online merge in split order (the running max raised, the
    // accumulated rows rescaled)
    constexpr int ZB = 4;
    float m = -INFINITY, l = 0.f;
    f32x16_t acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    for (int z0 = 0; z0 < NS; z0 += ZB) {
      u32x4_t ml[ZB], ov[ZB][4];
#pragma unroll
      for (int j = 0; j < ZB; ++j) {
        const int z = min(z0 + j, NS - 1);
        const uint32_t base = (uint32_t)(((size_t)bh * NS + z) * SPLIT_STATE) + lane * 16;
        ml[j] = __builtin_amdgcn_raw_buffer_load_b128(rp, base + 16 * 1024, 0, CPOL_SC1_A);
#pragma unroll
        for (int rq = 0; rq < 4; ++rq)
          ov[j][rq] = __builtin_amdgcn_raw_buffer_load_b128(rp, base + (ds * 4 + rq) * 1024, 0, CPOL_SC1_A);
      }
#pragma unroll
      for (int j = 0; j < ZB; ++j) {
        if (z0 + j >= NS) break;
        const float mz = __uint_as_float(ml[j][0]);
        if (mz == -INFINITY) continue;  // a split that saw no key adds nothing
        const float mn = fmaxf(m, mz);
        const float ar = m == -INFINITY ? 0.f : exp2_hw(m - mn), az = exp2_hw(mz - mn);
        m = mn;
        l = l * ar + __uint_as_float(ml[j][1]) * az;
#pragma unroll
        for (int rq = 0; rq < 4; ++rq)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[4 * rq + e] = acc[4 * rq + e] * ar + __uint_as_float(ov[j][rq][e]) * az;
      }
    }
    store_rows(&acc, ds, 1, l);
  }
  if (tid == 0) ticket[bh] = 0;
#endif
}

}  // namespace

size_t attn_split_bytes(int B, int Hq) { return (size_t)std::max(B * Hq, 512) * SPLIT_STATE; }

void launch_attn_bf16(const bf16_t* q, const bf16_t* k, const f16_t* vt, bf16_t* out, int B, int Lq, int L, int Hq,
                      int Hkv, hipStream_t s, float* split_part, int* split_ticket) {
  if (B * Lq == 0) return;
  if (Lq <= QW && split_part && split_ticket) {
    // one query group per head: the keys split over NS workgroups of 4 waves
    // when that fills 7/8 of the CUs, else of 2 waves (shorter sequences)
    const long bh = (long)B * Hq, cus = std::min(device_cu_count(), 512);
    const int nt = (L + KT2 - 1) / KT2;
    auto splits = [&](int nws) { return (int)std::max(1L, std::min<long>(cus / bh, (nt + nws - 1) / nws)); };
    const int ns4 = splits(4);
    if (8 * bh * ns4 >= 7 * cus || ns4 == 1) {
      hipLaunchKernelGGL(attn_split_kernel<4>, dim3(bh * ns4), dim3(256), 0, s, q, k, vt, out, split_part,
                         split_ticket, Lq, L, Hq, Hkv, ns4);
    } else {
      const int ns2 = splits(2);
      hipLaunchKernelGGL(attn_split_kernel<2>, dim3(bh * ns2), dim3(128), 0, s, q, k, vt, out, split_part,
                         split_ticket, Lq, L, Hq, Hkv, ns2);
    }
    DLLM_LAUNCH_CHECK("attn_split");
    return;
  }
  if (L % 8 == 0) {
    // streaming kernel: 8 waves (256 queries) per workgroup when that still gives
    // two or more workgroups per CU over the launch, else 4 waves; when even the
    // 4-wave grid leaves CUs without a workgroup, or there is only one 32-query
    // group per (sequence, head), the key-split kernel (four waves per query over
    // interleaved 32-key tiles)
    const bool wide = (long)((Lq + 255) / 256) * Hq * B >= 512;
    const size_t lds = 3 * (size_t)STAGE;
    const long cus = device_cu_count();
    if (Lq <= QW || ((long)((Lq + 127) / 128) * Hq * B < cus && L > KT)) {
      // 32 queries per workgroup for a single query group, else 64 when that
      // still fits the CUs, else 96
      auto go = [&](auto qgc) {
        constexpr int QG = decltype(qgc)::value;
        // merge: every wave's state and the staged rows (up to 64 queries), or
        // the three handed-over groups' states (96)
        constexpr size_t ring = 2 * (size_t)STEP2,
                         merge = QG <= 2 ? (size_t)QG * KGRP * 17 * 64 * 16 + (size_t)QG * QW * 272
                                         : (size_t)3 * QG * 17 * 64 * 16;
        constexpr size_t lds_kv = ring > merge ? ring : merge;
        static const hipError_t a = hipFuncSetAttribute((const void*)attn_kv4_kernel<QG>,
                                                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_kv);
        hip_check(a, "hipFuncSetAttribute(attn_kv4)");
        hipLaunchKernelGGL(attn_kv4_kernel<QG>, dim3(ceil_div(Lq, QW * QG) * Hq * B), dim3(64 * QG * KGRP), lds_kv, s,
                           q, k, vt, out, Lq, L, Hq, Hkv);
      };
      if (Lq <= QW)
        go(std::integral_constant<int, 1>{});
      else if ((long)ceil_div(Lq, QW * 2) * Hq * B <= cus)
        go(std::integral_constant<int, 2>{});
      else
        go(std::integral_constant<int, 3>{});
      DLLM_LAUNCH_CHECK("attn_kv4");
      return;
    }
    if (wide) {
      static const hipError_t a8 =
          hipFuncSetAttribute((const void*)attn_stream_kernel<8>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      hip_check(a8, "hipFuncSetAttribute(attn_stream<8>)");
      hipLaunchKernelGGL(attn_stream_kernel<8>, dim3(ceil_div(Lq, QW * 8) * Hq * B), dim3(512), lds, s, q, k, vt, out,
                         Lq, L, Hq, Hkv);
    } else {
      static const hipError_t a4 =
          hipFuncSetAttribute((const void*)attn_stream_kernel<4>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      hip_check(a4, "hipFuncSetAttribute(attn_stream<4>)");
      hipLaunchKernelGGL(attn_stream_kernel<4>, dim3(ceil_div(Lq, QW * 4) * Hq * B), dim3(256), lds, s, q, k, vt, out,
                         Lq, L, Hq, Hkv);
    }
    DLLM_LAUNCH_CHECK("attn_stream");
    return;
  }
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)attn_bf16_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, 2 * STAGE);
  hip_check(attr, "hipFuncSetAttribute(attn_bf16)");
  hipLaunchKernelGGL(attn_bf16_kernel, dim3(ceil_div(Lq, QW * NW) * Hq * B), dim3(256), 2 * STAGE, s, q, k, vt, out, Lq,
                     L, Hq, Hkv);
  DLLM_LAUNCH_CHECK("attn_bf16");
}

}  // namespace dllm
