// Top-t anchor selection, S = TopK(scores, t) per pair (Section 3.3).
//
// One workgroup per pair.  Scores become order-preserving uint32 keys
// (score_key).  A 4-pass, 8-bit radix select finds the key K* of the t-th
// largest element and how many elements equal to K* must be kept; a final
// pass over positions in ascending order keeps every key > K* and the
// lowest-indexed ties, using ballot prefix sums, so the output is ascending and
// bit-exact.
#include "common.hpp"

namespace arckv {

namespace {
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
}

__global__ void __launch_bounds__(kSelThreads) k_select_topt(const float *__restrict__ scores, int T, int t,
                                                             int32_t *__restrict__ anchors,
                                                             int32_t *__restrict__ anchor_of) {
  __shared__ uint32_t hist[kSelWaves][256];
  __shared__ uint32_t s_prefix, s_remaining;
  __shared__ uint32_t wave_tot[2][kSelWaves];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float *s = scores + (size_t)b * T;
  uint32_t prefix = 0, mask = 0, remaining = (uint32_t)t;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < kSelWaves * 256; i += kSelThreads) (&hist[0][0])[i] = 0;
    __syncthreads();
    for (int j = tid; j < T; j += kSelThreads) {
      uint32_t k = score_key(s[j]);
      if ((k & mask) == prefix) atomicAdd(&hist[wave][(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 256) {  // fold the per-wave histograms
      uint32_t c = 0;
      for (int w = 0; w < kSelWaves; ++w) c += hist[w][tid];
      hist[0][tid] = c;
    }
    __syncthreads();
    if (tid == 0) {   // walk digits from the top until `remaining` falls inside a bin
      uint32_t above = 0;
      int dg = 255;
      for (; dg > 0; --dg) {
        if (above + hist[0][dg] >= remaining) break;
        above += hist[0][dg];
      }
      s_prefix = prefix | ((uint32_t)dg << shift);
      s_remaining = remaining - above;
    }
    __syncthreads();
    prefix = s_prefix;
    remaining = s_remaining;
    mask |= 255u << shift;
    __syncthreads();
  }
  // prefix = K*, remaining = number of K*-ties to keep (lowest positions first)
  const uint32_t kstar = prefix;
  uint32_t eq_base = 0, out_base = 0;
  const uint64_t lanemask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int j0 = 0; j0 < T; j0 += kSelThreads) {
    const int j = j0 + tid;
    uint32_t k = j < T ? score_key(s[j]) : 0u;
    const bool in = j < T;
    const bool eq = in && k == kstar;
    uint64_t beq = __ballot(eq);
    uint32_t eq_rank_w = __popcll(beq & lanemask);
    if (lane == 0) wave_tot[0][wave] = __popcll(beq);
    __syncthreads();
    uint32_t eq_before = eq_base;
    for (int w = 0; w < wave; ++w) eq_before += wave_tot[0][w];
    uint32_t eq_rank = eq_before + eq_rank_w;
    const bool sel = in && (k > kstar || (eq && eq_rank < remaining));
    uint64_t bsel = __ballot(sel);
    if (lane == 0) wave_tot[1][wave] = __popcll(bsel);
    __syncthreads();
    uint32_t out_before = out_base;
    for (int w = 0; w < wave; ++w) out_before += wave_tot[1][w];
    uint32_t pos = out_before + __popcll(bsel & lanemask);
    if (sel && pos < (uint32_t)t) anchors[(size_t)b * t + pos] = j;
    if (anchor_of && in) anchor_of[(size_t)b * T + j] = sel ? (int32_t)pos : -1;
    uint32_t eq_tot = 0, sel_tot = 0;
    for (int w = 0; w < kSelWaves; ++w) { eq_tot += wave_tot[0][w]; sel_tot += wave_tot[1][w]; }
    eq_base += eq_tot;
    out_base += sel_tot;
    __syncthreads();
  }
}

hipError_t launch_select(const float *scores, int B, int T, int t, int32_t *anchors, int32_t *anchor_of,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_select_topt, dim3(B), dim3(kSelThreads), 0, s, scores, T, t, anchors, anchor_of);
  return hipGetLastError();
}

}  // namespace arckv
