// Confidence-aware commit for one denoising step (Algorithm 1's body, Boxes 2-7).
//
// One workgroup; wavefront b handles sequence b and lane p handles in-block
// position p (block length <= 64), so every state entry has a single writer
// and the per-step count eta is a ballot + popcount.  Order inside the step:
// threshold / budget commits, eta, low-yield counter, grinding fallback,
// no-mask check, flush of what is still masked when the block ends.
//
// Fixed-schedule baseline (fixed set): the wave commits its fixed_k masked
// positions of highest confidence (lowest position first on equal confidence;
// a NaN confidence ranks lowest), found by fixed_k butterfly reductions --
// none at a step whose k_t is 0 (steps past the block length when T exceeds
// it); no s, B or ell is kept.
//
// The word *all_done receives 1 when every sequence has finished the block,
// plus the bits of the step's error word (shifted up by one), which is then
// cleared; the same word tagged with the step's sequence number goes to the
// host's pinned flag when one is given.
#include "kernels.h"

namespace dllm {

__global__ void __launch_bounds__(1024) commit_kernel(CommitArgs a) {
  const int b = threadIdx.x >> 6;
  const int p = threadIdx.x & 63;
  __shared__ int fin[16];
  int finished = 1;
  if (b < a.B) {
    int ell = a.ell[b];
    int dn = a.done[b];
    if (a.t == 0) {  // step-zero init of the block
      ell = 0;
      dn = 0;
    }
    if (!dn) {
      const bool lane_on = p < a.bl;
      const int g = a.g0 + p;
      const size_t sg = (size_t)b * a.G + g;
      bool masked = false;
      float c = 0.f;
      int tok = 0, bud = 0;
      if (lane_on) {
        masked = a.commit_step[sg] < 0;
        c = a.conf[(size_t)b * a.bl + p];
        tok = a.argmax[(size_t)b * a.bl + p];
      }
      int why = 0;
      bool exit = false;
      if (a.fixed) {
        const float ce = c == c ? c : -INFINITY;
        bool sel = false;
        for (int it = 0; it < a.fixed_k; ++it) {
          int e = masked && !sel ? 1 : 0, bp = e ? p : 64;
          float bc = e ? ce : -INFINITY;
#pragma unroll
          for (int off = 32; off > 0; off >>= 1) {
            const int oe = __shfl_xor(e, off, 64), op = __shfl_xor(bp, off, 64);
            const float oc = __shfl_xor(bc, off, 64);
            if (oe > e || (oe == e && (oc > bc || (oc == bc && op < bp)))) {
              e = oe;
              bc = oc;
              bp = op;
            }
          }
          if (e == 0) break;  // nothing eligible is left (the same on every lane)
          if (p == bp) sel = true;
        }
        const bool remaining = masked && !sel;
        exit = __ballot(remaining) == 0ull;
        const bool flush = (exit || a.t == a.T - 1) && remaining;
        if (a.t == a.T - 1) exit = true;
        why = sel ? 5 : flush ? 4 : 0;
        ell = 0;
      } else {
        if (lane_on) {
          if (a.t == 0) {  // Box 2 (s_i = c_i^(0)) and Box 5 (budget tiers, top to bottom)
            if (c > a.s_easy && p < a.p_easy) bud = a.b_easy;
            else if (c < a.s_hard || p >= a.p_hard) bud = a.b_hard;
            else bud = a.b_mid;
            a.sv[sg] = c;
            a.budget[sg] = bud;
          } else {
            bud = a.budget[sg];
          }
        }
        const int band = (p >= a.edge[0]) + (p >= a.edge[1]) + (p >= a.edge[2]);
        const bool by_thr = masked && (c >= a.thr[band]);                         // Box 6 rule
        const bool by_bud = masked && !by_thr && a.budget_on && (a.t >= bud);   // Box 5 force
        const bool newly = by_thr || by_bud;
        const int eta = __popcll(__ballot(newly));
        ell = ((double)eta < a.eta_bar) ? ell + 1 : 0;                          // Box 7 counter
        bool forced = false;
        if (a.grind_on && ell >= a.patience) {                                  // grinding fallback
          forced = masked && !newly && (c > a.theta_fb);
          exit = true;
        }
        const bool remaining = masked && !newly && !forced;
        if (__ballot(remaining) == 0ull) exit = true;
        bool flush = false;
        if (exit || a.t == a.T - 1) {
          flush = remaining;
          exit = true;
        }
        why = by_thr ? 1 : by_bud ? 2 : forced ? 3 : flush ? 4 : 0;
      }
      if (why) {
        a.x[(size_t)b * a.L + a.P + g] = tok;
        a.commit_step[sg] = a.t;
        a.reason[sg] = (int8_t)why;
      }
      if (p == 0) {
        a.ell[b] = ell;
        a.done[b] = exit ? 1 : 0;
      }
      finished = exit ? 1 : 0;
    }
  }
  if (p == 0 && b < 16) fin[b] = finished;
  __syncthreads();
  if (threadIdx.x == 0) {
    int all = 1;
    for (int i = 0; i < a.B; ++i) all &= fin[i];
    int e = 0;
    if (a.err) {
      e = *a.err;
      *a.err = 0;
    }
    const int word = all | (e << 1);
    if (a.all_done) *a.all_done = word;
    // a vector store to host memory at system scope; relaxed: the word is all
    // the host reads before its next launch (device data it may read later
    // goes through stream-ordered copies)
    if (a.host_flag) __hip_atomic_store(a.host_flag, (a.seq << 8) | word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

void launch_commit(const CommitArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(commit_kernel, dim3(1), dim3(64 * a.B), 0, s, a);
  DLLM_LAUNCH_CHECK("commit");
}

}  // namespace dllm
