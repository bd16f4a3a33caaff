// Decode-time attention over a compacted block, optionally followed by an
// uncompressed block (eq. compact_attention; joint form of Appendix A.7,
// eq. concatenated_attention_preservation).  For pair p (one sequence and
// KV head) and each of its G query rows q:
//   o = softmax([s q C_k^T + beta, s q K_f^T]) [C_v; V_f]
// i.e. the fitted bias beta is added to the compact block's logits and the
// uncompressed block gets zero bias.  beta = NULL (zero bias) with C_k = K,
// C_v = V and F = 0 is plain full-cache attention.
//
// HBM-bound: every key and value row is read once.  Split-key ("flash
// decoding") in two kernels:
//   k_attend_partial  a workgroup of 8 waves takes 256 consecutive keys of
//                     the concatenated block; each wave scores its 32 keys
//                     against the G queries on MFMA 16x16x32 (keys as rows,
//                     queries as zero-padded columns), takes the softmax of
//                     its chunk, and accumulates P V on the VALU (each lane
//                     owns 8 dims of 4 interleaved keys, probabilities
//                     broadcast from LDS).  The eight waves' (max, sum, o) are
//                     merged in LDS into one partial per workgroup.  All of
//                     the chunk's K and V loads are issued up front.
//   k_attend_combine  merges the partials of a pair with the usual
//                     max-rescaling and writes o.
#include <mutex>

#include "common.hpp"

namespace arckv {

namespace {
constexpr int kAttKPW = 32;                 // keys per wave
constexpr int kAttW = 8;                    // waves per workgroup
constexpr int kAttChunk = kAttW * kAttKPW;  // keys per workgroup

typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

__device__ inline f32x4_t mfma16(bf16x8 a, bf16x8 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Row `key` of the concatenated block [compact (t rows); fixed (F rows)], or
// nullptr past the end.
__device__ inline const bf16 *att_row(const bf16 *C, const bf16 *Fx, int p, int t, int F, int key) {
  if (key < t) return C + ((size_t)p * t + key) * kHeadDim;
  if (key < t + F) return Fx + ((size_t)p * F + (key - t)) * kHeadDim;
  return nullptr;
}
}  // namespace

template <int G>
__global__ void __launch_bounds__(64 * kAttW) k_attend_partial(int t, int F, float scale, const bf16 *__restrict__ Q,
                                                         const bf16 *__restrict__ Ck, const float *__restrict__ beta,
                                                         const bf16 *__restrict__ Cv, const bf16 *__restrict__ Kf,
                                                         const bf16 *__restrict__ Vf, float *__restrict__ part_o,
                                                         float *__restrict__ part_ml, int nch) {
  static_assert(G >= 1 && G <= 8, "query rows per pair");
  __shared__ float sP[kAttW][kAttKPW][G];       // probabilities of each wave's keys
  __shared__ float sO[kAttW][G][kHeadDim];      // per-wave partial outputs
  __shared__ float sM[kAttW][G], sL[kAttW][G];
  const int p = blockIdx.y, ch = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = t + F;
  const int key0 = ch * kAttChunk + wave * kAttKPW;
  const int g = lane >> 4, r = lane & 15;        // MFMA lane coordinates

  // ---- issue every load of the chunk: K as MFMA A fragments (key rows), V rows
  // for the PV pass (lane = key group g (keys key0 + 4 i + g) x dims 8 r .. 8 r + 7)
  const bf16x8 zero8 = Mfma<bf16>::zero();
  constexpr int KT = kAttKPW / 16, VI = kAttKPW / 4;
  bf16x8 kf[KT][4];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    const bf16 *row = att_row(Ck, Kf, p, t, F, key0 + 16 * kt + r);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      kf[kt][ks] = row ? *reinterpret_cast<const bf16x8 *>(row + 32 * ks + 8 * g) : zero8;
  }
  bf16x8 vf[VI];
#pragma unroll
  for (int i = 0; i < VI; ++i) {
    const bf16 *row = att_row(Cv, Vf, p, t, F, key0 + 4 * i + g);
    vf[i] = row ? *reinterpret_cast<const bf16x8 *>(row + 8 * r) : zero8;
  }
  // queries as the B operand: column r = query row r (zero for r >= G)
  bf16x8 qf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
    qf[ks] = r < G ? *reinterpret_cast<const bf16x8 *>(Q + ((size_t)p * G + r) * kHeadDim + 32 * ks + 8 * g) : zero8;

  // ---- logits: lane (g, r) holds keys key0 + 16 kt + 4 g + j (j < 4) for query r
  float sv[VI];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) acc = mfma16(kf[kt][ks], qf[ks], acc);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int key = key0 + 16 * kt + 4 * g + j;
      float b = 0.0f;
      if (beta && key < t) b = beta[(size_t)p * t + key];
      sv[4 * kt + j] = key < L ? fmaf(scale, acc[j], b) : -INFINITY;
    }
  }
  // ---- softmax of the wave's keys per query (reduce the lane's VI, then over g)
  float m = sv[0];
#pragma unroll
  for (int i = 1; i < VI; ++i) m = fmaxf(m, sv[i]);
  m = fmaxf(m, __shfl_xor(m, 16, 64));
  m = fmaxf(m, __shfl_xor(m, 32, 64));
  const float mref = m == -INFINITY ? 0.0f : m;   // a wave past the end keeps zero mass
  float l = 0.0f;
#pragma unroll
  for (int i = 0; i < VI; ++i) {
    sv[i] = __expf(sv[i] - mref);
    l += sv[i];
  }
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (r < G) {
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int j = 0; j < 4; ++j) sP[wave][16 * kt + 4 * g + j][r] = sv[4 * kt + j];
    if (g == 0) {
      sM[wave][r] = m;
      sL[wave][r] = l;
    }
  }
  __syncthreads();
  // ---- P V: lane (g, r) accumulates keys 4 i + g, dims 8 r .. 8 r + 7
  float o[G][8];
#pragma unroll
  for (int q = 0; q < G; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[q][e] = 0.0f;
#pragma unroll
  for (int i = 0; i < VI; ++i) {
    float pq[G];
#pragma unroll
    for (int q = 0; q < G; ++q) pq[q] = sP[wave][4 * i + g][q];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float v = (float)vf[i][e];
#pragma unroll
      for (int q = 0; q < G; ++q) o[q][e] = fmaf(pq[q], v, o[q][e]);
    }
  }
#pragma unroll
  for (int q = 0; q < G; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float x = o[q][e];
      x += __shfl_xor(x, 16, 64);
      x += __shfl_xor(x, 32, 64);
      o[q][e] = x;
    }
  if (g == 0) {
#pragma unroll
    for (int q = 0; q < G; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) sO[wave][q][8 * r + e] = o[q][e];
  }
  __syncthreads();
  // ---- merge the waves: one partial (max, sum, o) per query for the chunk
  float *po = part_o + (((size_t)p * nch + ch) * G) * kHeadDim;
  float *pml = part_ml + (((size_t)p * nch + ch) * G) * 2;
  for (int idx = tid; idx < G * kHeadDim; idx += 64 * kAttW) {
    const int q = idx / kHeadDim, dim = idx % kHeadDim;
    float M = sM[0][q];
#pragma unroll
    for (int w = 1; w < kAttW; ++w) M = fmaxf(M, sM[w][q]);
    const float Mref = M == -INFINITY ? 0.0f : M;
    float acc = 0.0f, lsum = 0.0f;
#pragma unroll
    for (int w = 0; w < kAttW; ++w) {
      const float f = sM[w][q] == -INFINITY ? 0.0f : __expf(sM[w][q] - Mref);
      acc = fmaf(f, sO[w][q][dim], acc);
      lsum = fmaf(f, sL[w][q], lsum);
    }
    po[(size_t)q * kHeadDim + dim] = acc;
    if (dim == 0) {
      pml[2 * q] = M;
      pml[2 * q + 1] = lsum;
    }
  }
}

// One workgroup per pair: thread (q, dim) merges the pair's nch partials.
__global__ void __launch_bounds__(1024) k_attend_combine(int G, const float *__restrict__ part_o,
                                                          const float *__restrict__ part_ml, int nch,
                                                          float *__restrict__ out) {
  const int p = blockIdx.x, idx = threadIdx.x;
  if (idx >= G * kHeadDim) return;
  const int q = idx / kHeadDim, dim = idx % kHeadDim;
  const float *ml = part_ml + (size_t)p * nch * G * 2;
  // Both sweeps are unrolled so that eight chunks' loads are in flight at once
  // (one dependent load per chunk left the long contexts latency-bound).
  float M = -INFINITY;
#pragma unroll 8
  for (int c = 0; c < nch; ++c) M = fmaxf(M, ml[((size_t)c * G + q) * 2]);
  const float Mref = M == -INFINITY ? 0.0f : M;
  float acc = 0.0f, lsum = 0.0f;
  const float *po = part_o + (size_t)p * nch * G * kHeadDim;
#pragma unroll 8
  for (int c = 0; c < nch; ++c) {
    const float mc = ml[((size_t)c * G + q) * 2];
    const float f = mc == -INFINITY ? 0.0f : __expf(mc - Mref);
    acc = fmaf(f, po[((size_t)c * G + q) * kHeadDim + dim], acc);
    lsum = fmaf(f, ml[((size_t)c * G + q) * 2 + 1], lsum);
  }
  out[((size_t)p * G + q) * kHeadDim + dim] = acc / lsum;
}

int attend_chunks(int t, int F) { return (t + F + kAttChunk - 1) / kAttChunk; }

// ---------------------------------------------------------------- static scratch
// The split-key partials of arckv_attend_noalloc live in this file-scope
// device array instead of a caller workspace: one copy per GPU, held until the
// process ends.  On the host the array's name is only a stand-in, never a
// device address; the address is taken once per device with
// hipGetSymbolAddress (with that device current) and kept here.
constexpr size_t kAttendScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kAttendScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

size_t attend_scratch_bytes() { return kAttendScratchBytes; }

// Device address of the current device's scratch array.
hipError_t attend_scratch(void **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_attend(int P, int G, int t, int F, float scale, const void *Q, const void *Ck, const float *beta,
                         const void *Cv, const void *Kf, const void *Vf, float *part_o, float *part_ml, float *out,
                         hipStream_t s) {
  const int nch = attend_chunks(t, F);
  dim3 grid((unsigned)nch, (unsigned)P);
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, dim3(64 * kAttW), 0, s, t, F, scale, (const bf16 *)Q, (const bf16 *)Ck, beta,
                       (const bf16 *)Cv, (const bf16 *)Kf, (const bf16 *)Vf, part_o, part_ml, nch);
  };
  switch (G) {
    case 1: go(k_attend_partial<1>); break;
    case 2: go(k_attend_partial<2>); break;
    case 4: go(k_attend_partial<4>); break;
    case 8: go(k_attend_partial<8>); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_attend_combine, dim3((unsigned)P), dim3((unsigned)(G * kHeadDim)), 0, s, G, part_o, part_ml,
                     nch, out);
  return hipGetLastError();
}

}  // namespace arckv
