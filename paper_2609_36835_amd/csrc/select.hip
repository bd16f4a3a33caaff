// Top-t anchor selection, S = TopK(scores, t) per pair (Section 3.3), with the
// optional per-pair budgets of eq. per_head_budget and the chunked selection of
// Appendix A.3 (the union of each chunk's local top-t_c,
// t_c = clip_[1,T_c](round(t T_c / T)), rounded half up).
//
// One workgroup of 1024 threads per (pair, chunk).  Scores become order-preserving
// uint32 keys (score_key).  Lane l of wave w owns the KPT consecutive positions
// starting at (64 w + l) KPT, so positions ascend with (wave, lane, i).  When
// T <= 32768 the keys are read once, coalesced, through a padded LDS copy and
// then stay in registers; longer caches re-read them from memory (L2) on every
// pass.
//
// A 3-pass radix select (digits of 11, 11 and 10 bits from the top) finds the
// key K* of the t-th largest element and how many elements equal to K* must be
// kept (the lowest positions win ties): each pass histograms the keys that
// match the digits found so far, and a block-wide suffix scan over the bins
// picks the next digit.  The leading digit is wide because real-valued scores
// share their sign and leading exponent bits; a narrow one would send almost
// every key to a handful of bins, and same-address LDS atomics serialise.
// One block scan of the per-lane (greater, equal) counts then gives every lane
// its output offset, and each lane writes its selected positions in order, so
// the output is ascending and bit-exact.
#include "common.hpp"

namespace arckv {

namespace {
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelBins = 2048;   // widest digit: 11 bits
constexpr int kSelPasses = 3;
constexpr int kSelChunkThreshold = 10000;   // chunked selection applies when T > 10,000

// Anchors kept by a chunk of length Tc out of T for a pair budget tb; computed
// in double exactly as on the host, so both agree on every rounding.
__device__ inline int chunk_budget(int tb, int T, int Tc) {
  const int v = (int)floor((double)tb * (double)Tc / (double)T + 0.5);
  return min(Tc, max(1, v));
}

// Digit p of the key (from the top): bits [shift, shift + width).
__device__ inline int sel_shift(int p) { return p == 0 ? 21 : p == 1 ? 10 : 0; }
__device__ inline int sel_width(int p) { return p == 2 ? 10 : 11; }

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ inline uint32_t wave_incl_scan(uint32_t v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(v, off, 64);
    v += lane >= off ? o : 0u;
  }
  return v;
}
}  // namespace

struct SelArgs {
  int T;                   // positions per pair
  int t;                   // budget of every pair (when t_pair is null)
  const int32_t *t_pair;   // per-pair budgets [B] (device), or null
  int chunk_len;           // chunk length when nchunks > 1
  int nchunks;             // chunks per pair (1 = global top-t)
  int t_stride;            // row length of the anchors output
};

// KPT: keys per lane held in registers (chunk length <= 1024 KPT); 0 = read from memory.
template <int KPT>
__global__ void __launch_bounds__(kSelThreads) k_select_topt(const float *__restrict__ scores, SelArgs a,
                                                             int32_t *__restrict__ anchors) {
  extern __shared__ uint32_t sel_keys[];   // [Tc + Tc/32] padded key copy (KPT > 0)
  __shared__ uint32_t hist[kSelBins];
  __shared__ uint32_t s_wtot[2][kSelWaves];
  __shared__ uint32_t s_prefix, s_remaining;
  const int b = blockIdx.x / a.nchunks, chunk = blockIdx.x % a.nchunks;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // this workgroup's segment [seg0, seg0 + T) of the pair and its budget t
  const int tb = a.t_pair ? min(max(a.t_pair[b], 1), a.T) : a.t;
  const int seg0 = chunk * a.chunk_len;
  const int T = a.nchunks > 1 ? min(a.chunk_len, a.T - seg0) : a.T;
  const int t = a.nchunks > 1 ? chunk_budget(tb, a.T, T) : tb;
  int off = 0;   // anchors kept by the earlier chunks of the pair
  for (int c = 0; c < chunk; ++c) off += chunk_budget(tb, a.T, min(a.chunk_len, a.T - c * a.chunk_len));
  const float *s = scores + (size_t)b * a.T + seg0;
  const int per = KPT > 0 ? KPT : (T + kSelThreads - 1) / kSelThreads;   // positions per lane
  const int p0 = tid * per;
  uint32_t kr[KPT > 0 ? KPT : 1];
  if constexpr (KPT > 0) {
    // position p lives at LDS word p + p / 32, so both the coalesced fill and
    // the per-lane reads of 32 consecutive positions are free of bank conflicts
    for (int p = tid; p < T; p += kSelThreads) sel_keys[p + (p >> 5)] = score_key(s[p]);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int p = p0 + i;
      kr[i] = p < T ? sel_keys[p + (p >> 5)] : 0u;
    }
  }
  // f(key, position, valid) over this lane's positions in ascending order
  auto for_each = [&](auto &&f) {
    if constexpr (KPT > 0) {
#pragma unroll
      for (int i = 0; i < KPT; ++i) f(kr[i], p0 + i, p0 + i < T);
    } else {
      for (int i = 0; i < per; ++i) {
        const int p = p0 + i;
        const bool v = p < T;
        f(v ? score_key(s[p]) : 0u, p, v);
      }
    }
  };

  uint32_t prefix = 0, mask = 0, remaining = (uint32_t)t;
  for (int pass = 0; pass < kSelPasses; ++pass) {
    const int shift = sel_shift(pass);
    const uint32_t dmask = (1u << sel_width(pass)) - 1u;
    for (int i = tid; i < kSelBins; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    for_each([&](uint32_t k, int, bool v) {
      if (v && (k & mask) == prefix) atomicAdd(&hist[(k >> shift) & dmask], 1u);
    });
    __syncthreads();
    // thread i holds digits d_hi = 2047 - 2i and d_lo = 2046 - 2i; the inclusive
    // scan over i counts the matching keys with digit >= d_lo
    const int d_hi = kSelBins - 1 - 2 * tid, d_lo = d_hi - 1;
    const uint32_t c_hi = hist[d_hi], c_lo = hist[d_lo], c = c_hi + c_lo;
    uint32_t incl = wave_incl_scan(c, lane);
    if (lane == 63) s_wtot[0][wave] = incl;
    __syncthreads();
    for (int w = 0; w < wave; ++w) incl += s_wtot[0][w];
    // exactly one thread has (keys above its digits) < remaining <= (keys at or above them)
    const uint32_t above = incl - c;
    if (incl >= remaining && above < remaining) {
      const bool hi = above + c_hi >= remaining;
      s_prefix = prefix | ((uint32_t)(hi ? d_hi : d_lo) << shift);
      s_remaining = remaining - (hi ? above : above + c_hi);
    }
    __syncthreads();
    prefix = s_prefix;
    remaining = s_remaining;
    mask |= dmask << shift;
  }
  // prefix = K*; keep every key > K* and the first `remaining` keys == K*
  const uint32_t kstar = prefix;
  uint32_t gt = 0, eq = 0;
  for_each([&](uint32_t k, int, bool v) {
    gt += v && k > kstar;
    eq += v && k == kstar;
  });
  const uint32_t gt_in = wave_incl_scan(gt, lane), eq_in = wave_incl_scan(eq, lane);
  if (lane == 63) {
    s_wtot[0][wave] = gt_in;
    s_wtot[1][wave] = eq_in;
  }
  __syncthreads();
  uint32_t gt_before = gt_in - gt, eq_before = eq_in - eq;
  for (int w = 0; w < wave; ++w) {
    gt_before += s_wtot[0][w];
    eq_before += s_wtot[1][w];
  }
  uint32_t out = gt_before + min(eq_before, remaining);
  uint32_t eq_seen = eq_before;
  int32_t *dst = anchors + (size_t)b * a.t_stride;
  const uint32_t lim = (uint32_t)min(off + t, a.t_stride);   // off + out < off + t by construction
  out += (uint32_t)off;
  for_each([&](uint32_t k, int p, bool v) {
    const bool is_eq = v && k == kstar;
    const bool sel = v && (k > kstar || (is_eq && eq_seen < remaining));
    if (sel && out < lim) dst[out] = seg0 + p;
    out += sel;
    eq_seen += is_eq;
  });
  // the pair's last chunk pads its row past the realised count
  if (chunk == a.nchunks - 1)
    for (int i = off + t + tid; i < a.t_stride; i += kSelThreads) dst[i] = -1;
}

// chunk_len <= 0 or T <= 10000: global top-t.  t_pair (device, nullable)
// overrides t per pair; rows of `anchors` are t_stride long, padded with -1.
hipError_t launch_select_ex(const float *scores, int B, int T, int t, const int32_t *t_pair, int chunk_len,
                            int t_stride, int32_t *anchors, hipStream_t s) {
  SelArgs a;
  a.T = T;
  a.t = t;
  a.t_pair = t_pair;
  a.nchunks = (chunk_len > 0 && T > kSelChunkThreshold) ? (T + chunk_len - 1) / chunk_len : 1;
  a.chunk_len = a.nchunks > 1 ? chunk_len : T;
  a.t_stride = t_stride;
  const int seg = a.nchunks > 1 ? a.chunk_len : T;
  const int per_lane = (seg + kSelThreads - 1) / kSelThreads;
  auto go = [&](auto kern, bool cached) {
    const size_t lds = cached ? (size_t)(seg + seg / 32 + 1) * sizeof(uint32_t) : 0;
    if (lds > 48 * 1024) {
      hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)(B * a.nchunks)), dim3(kSelThreads), lds, s, scores, a, anchors);
    return hipGetLastError();
  };
  if (per_lane <= 8) return go(k_select_topt<8>, true);
  if (per_lane <= 16) return go(k_select_topt<16>, true);
  if (per_lane <= 32) return go(k_select_topt<32>, true);
  return go(k_select_topt<0>, false);
}

hipError_t launch_select(const float *scores, int B, int T, int t, int32_t *anchors, hipStream_t s) {
  return launch_select_ex(scores, B, T, t, nullptr, 0, t, anchors, s);
}

}  // namespace arckv
