// The value-aware indexer of Appendix A.1 and its pooled scores (eq.
// indexer_pooling), for H_I = 8 index heads of width d_I = 128 and a value
// head of width d_A = 128 (bf16 operands, fp32 accumulation):
//
//   k_dsa_proj      out = N?(X1 W1^T + X2 W2^T) per 128-wide output block:
//                   the value head's projections U_q q, U_k k, U_v v (one
//                   block, no norm) and qbar = N(L_q q + L_c c),
//                   kbar = N(L_k k + L_v v) (eight blocks, RMS-normalised),
//                   eq. indexer_projection.  Output columns are the MFMA rows,
//                   so each lane owns one input row and the RMS reduction stays
//                   in the lane (plus one cross-half shuffle).
//   k_dsa_w         w_r = L_x x_r + b_x, one wave per reference position.
//   (value context) c = softmax(s_A (U_q Q)(U_k K)^T)(U_v V) is the row
//                   statistics kernel run on the projected cache (eq. value_context).
//   k_dsa_index     I_ij = sum_a w_ia LeakyReLU(qbar_ia . kbar_ja / sqrt(d_I))
//                   (eq. pairwise_index_score) for 64 queries per workgroup,
//                   whose qbar rows stay in LDS while the workgroup sweeps all
//                   keys (eight waves, two per SIMD so that one wave's
//                   LeakyReLU epilogue overlaps the other's MFMAs; each wave 32
//                   keys of a 256-key block, the next heads' key fragments
//                   prefetched during the current ones).  Pass 1
//                   keeps each row's softmax max and sum; pass 2 adds
//                   pi_ij^2 = exp(2 (I_ij - z_i)) / m_i^2 over the workgroup's
//                   queries into a per-(query block, key) partial.
//   k_dsa_pool      s_j = sqrt(sum of the partials / n).
#include "common.hpp"

namespace arckv {

namespace {
constexpr int kDsaH = 8;            // index heads H_I
constexpr int kDsaW = 128;          // d_I = d_A
constexpr int kDsaQB = 64;          // queries per index workgroup
constexpr int kDsaWaves = 8;        // index workgroup: 8 waves (two per SIMD) share one LDS query block
constexpr int kDsaKT = 1;           // 32-key tiles per wave (each LDS query fragment feeds kDsaKT MFMAs)
constexpr int kDsaKB = kDsaWaves * 32 * kDsaKT;   // keys per sweep step
constexpr float kLeaky = 0.1f;
constexpr float kRmsEps = 1e-6f;

__device__ inline bf16x8 load_frag(const bf16 *p) { return *reinterpret_cast<const bf16x8 *>(p); }
__device__ inline bf16x8 load_frag(const float *p) {
  const f32x4 a = *reinterpret_cast<const f32x4 *>(p), b = *reinterpret_cast<const f32x4 *>(p + 4);
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    r[e] = (bf16)a[e];
    r[4 + e] = (bf16)b[e];
  }
  return r;
}
}  // namespace

// out[p][row][a 128 + c] for rows < nrows; grid (ceil(nrows / 128), n_blocks, B).
// X1 [B][nrows][128] bf16; X2 (nullable) [B][nrows][128] of X2T; W1, W2
// [B][n_blocks 128][128] bf16.
template <typename X2T, bool NORM>
__global__ void __launch_bounds__(256) k_dsa_proj(const bf16 *__restrict__ X1, const X2T *__restrict__ X2,
                                                  const bf16 *__restrict__ W1, const bf16 *__restrict__ W2,
                                                  int nrows, int n_blocks, bf16 *__restrict__ out) {
  const int p = blockIdx.z, a = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int row = blockIdx.x * 128 + wave * 32 + col;
  const bool valid = row < nrows;
  const size_t xoff = ((size_t)p * nrows + (valid ? row : 0)) * kDsaW + 8 * h;
  const size_t woff = ((size_t)p * n_blocks * kDsaW + (size_t)a * kDsaW) * kDsaW + 8 * h;
  f32x16 acc[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) acc[mt] = zero16();
  for (int src = 0; src < (X2 ? 2 : 1); ++src) {
    const bf16 *W = src == 0 ? W1 : W2;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const bf16x8 xb = src == 0 ? load_frag(X1 + xoff + 16 * ks) : load_frag(X2 + xoff + 16 * ks);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
        acc[mt] = Mfma<bf16>::mma(load_frag(W + woff + (size_t)(32 * mt + col) * kDsaW + 16 * ks), xb, acc[mt]);
    }
  }
  // lane (h, col): input row `row`, output columns 32 mt + 8 g + 4 h + e
  float sc = 1.0f;
  if (NORM) {
    float ss = 0.0f;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int v = 0; v < 16; ++v) ss = fmaf(acc[mt][v], acc[mt][v], ss);
    ss += __shfl_xor(ss, 32, 64);
    sc = 1.0f / sqrtf(ss / (float)kDsaW + kRmsEps);
  }
  if (!valid) return;
  bf16 *o = out + ((size_t)p * nrows + row) * ((size_t)n_blocks * kDsaW) + (size_t)a * kDsaW + 4 * h;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = (bf16)(acc[mt][4 * g + e] * sc);
      *reinterpret_cast<bf16x4 *>(o + 32 * mt + 8 * g) = v;
    }
}

// w[p][r][a] = L_x[p][a] . x_{(p_off + p) / x_group, r} + b_x[p][a]; grid (n_pos, B), one wave.
__global__ void __launch_bounds__(64) k_dsa_w(const bf16 *__restrict__ X, const bf16 *__restrict__ Lx,
                                              const float *__restrict__ bx, int n_pos, int dx, int x_group,
                                              int p_off, float *__restrict__ w) {
  const int p = blockIdx.y, r = blockIdx.x, lane = threadIdx.x;
  const bf16 *x = X + ((size_t)((p_off + p) / x_group) * n_pos + r) * dx;
  const bf16 *L = Lx + (size_t)p * kDsaH * dx;
  float acc[kDsaH];
#pragma unroll
  for (int a = 0; a < kDsaH; ++a) acc[a] = 0.0f;
  for (int c = lane; c < dx; c += 64) {
    const float xv = (float)x[c];
#pragma unroll
    for (int a = 0; a < kDsaH; ++a) acc[a] = fmaf((float)L[(size_t)a * dx + c], xv, acc[a]);
  }
#pragma unroll
  for (int a = 0; a < kDsaH; ++a) {
    const float s = wave_sum(acc[a]);
    if (lane == 0) w[((size_t)p * n_pos + r) * kDsaH + a] = s + bx[p * kDsaH + a];
  }
}

// PASS 1: z[p][q], m[p][q] (softmax max and sum of row q over the keys).
// PASS 2: part[p][qblk][j] = sum over the block's queries of exp(2 (I - z)) / m^2.
// grid (ceil(n / 64), B); LDS: the block's qbar rows [64][1024] bf16 (16-byte
// chunks swizzled within each head's 256-byte run), w and the row statistics.
template <int PASS>
__global__ void __launch_bounds__(64 * kDsaWaves) __attribute__((amdgpu_waves_per_eu(2, 2))) k_dsa_index(const bf16 *__restrict__ qbar, const bf16 *__restrict__ kbar,
                                                   const float *__restrict__ wpos, int n, int n_pos, int T,
                                                   float *__restrict__ z, float *__restrict__ m,
                                                   float *__restrict__ part) {
  extern __shared__ __attribute__((aligned(16))) char dsa_smem[];
  char *sq = dsa_smem;                                                  // 64 x 2048 B
  float *sw = reinterpret_cast<float *>(dsa_smem + kDsaQB * 2048);     // [64][8]
  float *sred = sw + kDsaQB * kDsaH;                                    // [waves][64][2]
  const int p = blockIdx.y, q0 = blockIdx.x * kDsaQB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const float inv_sqrt = 1.0f / sqrtf((float)kDsaW);
  // ---- stage qbar rows (missing rows read as zero) and the head weights w / sqrt(d_I)
  for (int e = tid; e < kDsaQB * 128; e += 64 * kDsaWaves) {
    const int q = e >> 7, c = e & 127;
    bf16x8 v = Mfma<bf16>::zero();
    if (q0 + q < n) v = load_frag(qbar + ((size_t)p * n + q0 + q) * (kDsaH * kDsaW) + 8 * c);
    const int phys = (c & ~15) | ((c ^ q) & 15);
    *reinterpret_cast<bf16x8 *>(sq + q * 2048 + phys * 16) = v;
  }
  for (int e = tid; e < kDsaQB * kDsaH; e += 64 * kDsaWaves) {
    const int q = e / kDsaH, a = e % kDsaH;
    sw[e] = q0 + q < n ? wpos[((size_t)p * n_pos + (q0 + q) % n_pos) * kDsaH + a] * inv_sqrt : 0.0f;
  }
  __syncthreads();
  float zq[2], im2[2];   // PASS 2: the row statistics of this lane's query columns
  if (PASS == 2) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int q = q0 + 32 * nt + col;
      zq[nt] = q < n ? z[(size_t)p * n + q] : 0.0f;
      const float mm = q < n ? m[(size_t)p * n + q] : 1.0f;
      im2[nt] = q < n ? 1.0f / (mm * mm) : 0.0f;
    }
  }
  float run_m[2] = {-INFINITY, -INFINITY}, run_s[2] = {0.0f, 0.0f};   // PASS 1
  const bf16 *kb = kbar + (size_t)p * T * (kDsaH * kDsaW) + 8 * h;
  const int nkb = (T + kDsaKB - 1) / kDsaKB;
  // a ring of two heads' key fragments for the wave's key tiles (128 VGPRs):
  // head a's slot is refilled with head a + 2 (or, for the last two heads, the
  // next block's first two) right after use, so every load has a head of MFMAs
  // to land
  constexpr int RING = 2;
  bf16x8 af[RING][kDsaKT][8];
  auto fetch = [&](int kbk_, int a, bf16x8 (&f)[kDsaKT][8]) {
#pragma unroll
    for (int kt = 0; kt < kDsaKT; ++kt) {
      const int key = kbk_ * kDsaKB + wave * (32 * kDsaKT) + 32 * kt + col;
      const bf16 *krow = kb + (size_t)(key < T ? key : 0) * (kDsaH * kDsaW) + a * kDsaW;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) f[kt][ks] = key < T ? load_frag(krow + 16 * ks) : Mfma<bf16>::zero();
    }
  };
#pragma unroll
  for (int a = 0; a < RING; ++a) fetch(0, a, af[a]);
  for (int kbk = 0; kbk < nkb; ++kbk) {
    // the query embeddings are re-read from LDS in every key block (not held in registers)
    asm volatile("" ::: "memory");
    float I[2][kDsaKT][16];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int kt = 0; kt < kDsaKT; ++kt)
#pragma unroll
        for (int v = 0; v < 16; ++v) I[nt][kt][v] = 0.0f;
#pragma unroll 1
    for (int a0 = 0; a0 < kDsaH; a0 += RING) {
      asm volatile("" ::: "memory");
#pragma unroll
      for (int i = 0; i < RING; ++i) {
        const int a = a0 + i;
        // head a: S = kbar_a qbar_a^T for both query tiles and every key tile,
        // I += (w_a / sqrt d_I) LeakyReLU(S); each query fragment read from LDS
        // serves all key tiles
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int q = 32 * nt + col;
          f32x16 acc[kDsaKT];
#pragma unroll
          for (int kt = 0; kt < kDsaKT; ++kt) acc[kt] = zero16();
#pragma unroll
          for (int ks = 0; ks < 8; ++ks) {
            const int c = 16 * a + 2 * ks + h;
            const int phys = (c & ~15) | ((c ^ q) & 15);
            const bf16x8 qf = *reinterpret_cast<const bf16x8 *>(sq + q * 2048 + phys * 16);
#pragma unroll
            for (int kt = 0; kt < kDsaKT; ++kt) acc[kt] = Mfma<bf16>::mma(af[i][kt][ks], qf, acc[kt]);
          }
          // w LeakyReLU(x) = w (1 + slope)/2 x + w (1 - slope)/2 |x|: two FMAs, |x| a free operand modifier
          const float wa = sw[q * kDsaH + a];
          const float wp = wa * (0.5f * (1.0f + kLeaky)), wn = wa * (0.5f * (1.0f - kLeaky));
#pragma unroll
          for (int kt = 0; kt < kDsaKT; ++kt)
#pragma unroll
            for (int v = 0; v < 16; ++v) I[nt][kt][v] = fmaf(wn, fabsf(acc[kt][v]), fmaf(wp, acc[kt][v], I[nt][kt][v]));
        }
        // refill the slot: head a + RING of this block, or the next block's head a + RING - H
        if (a + RING < kDsaH) fetch(kbk, a + RING, af[i]);
        else if (kbk + 1 < nkb) fetch(kbk + 1, a + RING - kDsaH, af[i]);
      }
    }
    // lane (h, col): keys kbk kDsaKB + 32 (kDsaKT wave + kt) + 8 g + 4 h + e, query column 32 nt + col
    const int kbase = kbk * kDsaKB + wave * (32 * kDsaKT) + 4 * h;
    auto key_of = [&](int kt, int v) { return kbase + 32 * kt + 8 * (v >> 2) + (v & 3); };
    if (PASS == 1) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        float tm = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < kDsaKT; ++kt)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (key_of(kt, v) < T) tm = fmaxf(tm, I[nt][kt][v]);
        const float nm = fmaxf(run_m[nt], tm);
        float ts = 0.0f;
#pragma unroll
        for (int kt = 0; kt < kDsaKT; ++kt)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (key_of(kt, v) < T) ts += __expf(I[nt][kt][v] - nm);
        run_s[nt] = (run_m[nt] == -INFINITY ? 0.0f : run_s[nt] * __expf(run_m[nt] - nm)) + ts;
        run_m[nt] = nm;
      }
    } else {
      // pi^2 summed over this workgroup's 64 queries, per key
      float *pp = part + ((size_t)p * gridDim.x + blockIdx.x) * T;
#pragma unroll
      for (int kt = 0; kt < kDsaKT; ++kt) {
        float cs[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float x = 0.0f;
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) x += __expf(2.0f * (I[nt][kt][v] - zq[nt])) * im2[nt];
          cs[v] = x;
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float x = cs[v];
#pragma unroll
          for (int o = 1; o < 32; o <<= 1) x += __shfl_xor(x, o, 64);
          cs[v] = x;
        }
        if (col == 0) {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int k = key_of(kt, v);
            if (k < T) pp[k] = cs[v];
          }
        }
      }
    }
  }
  if (PASS == 1) {
    // merge the two halves of the wave (they hold different keys), then the four waves
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const float om = __shfl_xor(run_m[nt], 32, 64), os = __shfl_xor(run_s[nt], 32, 64);
      const float nm = fmaxf(run_m[nt], om);
      const float s = (run_m[nt] == -INFINITY ? 0.0f : run_s[nt] * __expf(run_m[nt] - nm)) +
                      (om == -INFINITY ? 0.0f : os * __expf(om - nm));
      if (h == 0) {
        sred[(wave * kDsaQB + 32 * nt + col) * 2] = nm;
        sred[(wave * kDsaQB + 32 * nt + col) * 2 + 1] = s;
      }
    }
    __syncthreads();
    if (tid < kDsaQB && q0 + tid < n) {
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kDsaWaves; ++w) M = fmaxf(M, sred[(w * kDsaQB + tid) * 2]);
      float S = 0.0f;
#pragma unroll
      for (int w = 0; w < kDsaWaves; ++w) {
        const float mw = sred[(w * kDsaQB + tid) * 2];
        if (mw != -INFINITY) S += sred[(w * kDsaQB + tid) * 2 + 1] * __expf(mw - M);
      }
      z[(size_t)p * n + q0 + tid] = M;
      m[(size_t)p * n + q0 + tid] = S;
    }
  }
}

// s[p][j] = sqrt(sum over query blocks of part / n); grid (ceil(T / 256), B).
__global__ void __launch_bounds__(256) k_dsa_pool(const float *__restrict__ part, int nqb, int n, int T,
                                                  float *__restrict__ s) {
  const int p = blockIdx.y, j = blockIdx.x * 256 + threadIdx.x;
  if (j >= T) return;
  float acc = 0.0f;
  for (int b = 0; b < nqb; ++b) acc += part[((size_t)p * nqb + b) * T + j];
  s[(size_t)p * T + j] = sqrtf(acc / (float)n);
}

hipError_t launch_dsa_proj(const void *X1, const void *X2, bool x2_f32, const void *W1, const void *W2, int B,
                           int nrows, int n_blocks, bool norm, void *out, hipStream_t s) {
  dim3 grid((unsigned)((nrows + 127) / 128), (unsigned)n_blocks, (unsigned)B);
  auto o = (bf16 *)out;
  if (!X2) {
    if (norm) hipLaunchKernelGGL((k_dsa_proj<bf16, true>), grid, dim3(256), 0, s, (const bf16 *)X1,
                                 (const bf16 *)nullptr, (const bf16 *)W1, (const bf16 *)nullptr, nrows, n_blocks, o);
    else hipLaunchKernelGGL((k_dsa_proj<bf16, false>), grid, dim3(256), 0, s, (const bf16 *)X1,
                            (const bf16 *)nullptr, (const bf16 *)W1, (const bf16 *)nullptr, nrows, n_blocks, o);
  } else if (x2_f32) {
    hipLaunchKernelGGL((k_dsa_proj<float, true>), grid, dim3(256), 0, s, (const bf16 *)X1, (const float *)X2,
                       (const bf16 *)W1, (const bf16 *)W2, nrows, n_blocks, o);
  } else {
    hipLaunchKernelGGL((k_dsa_proj<bf16, true>), grid, dim3(256), 0, s, (const bf16 *)X1, (const bf16 *)X2,
                       (const bf16 *)W1, (const bf16 *)W2, nrows, n_blocks, o);
  }
  return hipGetLastError();
}

hipError_t launch_dsa_w(const void *X, const void *Lx, const float *bx, int B, int n_pos, int dx, int x_group,
                        int p_off, float *w, hipStream_t s) {
  hipLaunchKernelGGL(k_dsa_w, dim3((unsigned)n_pos, (unsigned)B), dim3(64), 0, s, (const bf16 *)X, (const bf16 *)Lx,
                     bx, n_pos, dx, x_group, p_off, w);
  return hipGetLastError();
}

size_t dsa_index_lds() {
  return (size_t)kDsaQB * 2048 + (size_t)kDsaQB * kDsaH * 4 + (size_t)kDsaWaves * kDsaQB * 2 * 4;
}
int dsa_query_blocks(int n) { return (n + kDsaQB - 1) / kDsaQB; }

hipError_t launch_dsa_index(int pass, const void *qbar, const void *kbar, const float *w, int B, int n, int n_pos,
                            int T, float *z, float *m, float *part, hipStream_t s) {
  dim3 grid((unsigned)dsa_query_blocks(n), (unsigned)B);
  const size_t lds = dsa_index_lds();
  auto k1 = k_dsa_index<1>;
  auto k2 = k_dsa_index<2>;
  hipError_t e = hipFuncSetAttribute((const void *)(pass == 1 ? k1 : k2),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  if (pass == 1)
    hipLaunchKernelGGL(k1, grid, dim3(64 * kDsaWaves), lds, s, (const bf16 *)qbar, (const bf16 *)kbar, w, n, n_pos, T, z, m,
                       part);
  else
    hipLaunchKernelGGL(k2, grid, dim3(64 * kDsaWaves), lds, s, (const bf16 *)qbar, (const bf16 *)kbar, w, n, n_pos, T, z, m,
                       part);
  return hipGetLastError();
}

hipError_t launch_dsa_pool(const float *part, int B, int n, int T, float *scores, hipStream_t s) {
  hipLaunchKernelGGL(k_dsa_pool, dim3((unsigned)((T + 255) / 256), (unsigned)B), dim3(256), 0, s, part,
                     dsa_query_blocks(n), n, T, scores);
  return hipGetLastError();
}

}  // namespace arckv
