// TOVA prompt compression for gfx950.  Section 2.1 names TOVA among the composed rule
// families: it evicts by the attention of the current query.  Appendix C runs the standalone
// TOVA baseline in prefill as well as decode; at the end of prefill the current query is the
// prompt's last one (position L - 1), so per (sequence, layer, KV head) job
//   S[j] = (1/G) sum_g softmax_j(q[hG+g, L-1] . k[j] / sqrt(d)),   j = 0 .. L-1,
// and the shared select and gather kernels keep the top-b of [0, L) (nothing forced).
//
// tova_logits_kernel<G>: one workgroup per (TOVA job, 128-key slice).  16 lanes per key row,
//   16 bytes each, so one wave load instruction reads four whole 256-byte rows; every lane
//   keeps its 16-byte piece of the G query rows as fp32, and the G dot products of a row are
//   summed over its 16 lanes (one DPP row) with four rotations.  The logits, scaled to log2
//   units, go to the workspace through LDS (coalesced rows), and the slice leaves its per-head
//   (max, sum of exp2(x - max)).  This is a matrix-vector product of G rows: HBM-bound on the
//   key stream, so it stays on the vector ALUs.
// tova_scores_kernel<G>: one workgroup per job and kTovaScoreKeys keys.  Each head's slice
//   pairs fold into (M_g, Z_g) by an online combination (exact: no fixed reference, nothing can
//   overflow; every workgroup of a job folds them in the same order); then
//   S[j] = (1/G) sum_g exp2(x_gj - M_g) / Z_g over the workgroup's keys.
// Sums run in a fixed order, so results are reproducible.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "rkv_internal.h"

namespace rkv {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kTovaThreads = 256;
constexpr int kKeysPerPass = kTovaThreads / 16;      // 16 key rows per pass of the workgroup
constexpr int kPasses = kSlice / kKeysPerPass;       // 8 passes cover a 128-key slice
constexpr int kTovaScoreKeys = 2048;                 // keys per score workgroup (8 per thread)

template <int CTRL>
__device__ __forceinline__ float dpp_rot(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}

// Combination of two (max, sum of exp2(x - max)) pairs.
__device__ __forceinline__ void combine(float& m, float& z, float m2, float z2) {
  const float M = fmaxf(m, m2);
  z = z * __builtin_amdgcn_exp2f(m - M) + z2 * __builtin_amdgcn_exp2f(m2 - M);
  m = M;
}

// First global job index of the TOVA slots (window-scored and full-span slots come first).
__device__ __forceinline__ int tova_job0(const PrefillLaunch& P) {
  return (P.n_window + P.n_full) * P.batch * P.n_kv_heads;
}

template <int G>
__global__ __launch_bounds__(kTovaThreads) void tova_logits_kernel(const PrefillLaunch P) {
  __shared__ float sX[G][kSlice];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = tid & 15, r = tid >> 4;
  const int L = P.seq_len, w = P.window, Hq = P.n_q_heads, Hkv = P.n_kv_heads, B = P.batch;
  const int nsl = P.n_slices;
  const int jt = blockIdx.x / nsl, slice = blockIdx.x - jt * nsl;
  const int job = tova_job0(P) + jt;
  const int h = job % Hkv, s = (job / Hkv) % B, slot = job / (Hkv * B);
  const PrefillLayer& ly = P.layer[slot];
  const int key0 = slice * kSlice;

  // the key rows of this thread's passes (keys past the prompt read row L - 1; unused)
  const uint16_t* khead = ly.k + (size_t)(s * Hkv + h) * L * kHeadDim;
  u32x4 kv[kPasses];
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    const int key = min(key0 + kKeysPerPass * p + r, L - 1);
    kv[p] = *reinterpret_cast<const u32x4*>(khead + (size_t)key * kHeadDim + 8 * c);
  }
  // this lane's 16-byte piece of each head's last-position query, as fp32
  float qf[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const u32x4 qv =
        *reinterpret_cast<const u32x4*>(ly.q + ((size_t)(s * Hq + h * G + g) * w + (w - 1)) * kHeadDim + 8 * c);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      qf[g][2 * u] = __uint_as_float(qv[u] << 16);
      qf[g][2 * u + 1] = __uint_as_float(qv[u] & 0xffff0000u);
    }
  }
  const float sl2 = P.scale_log2;
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    float kf[8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      kf[2 * u] = __uint_as_float(kv[p][u] << 16);
      kf[2 * u + 1] = __uint_as_float(kv[p][u] & 0xffff0000u);
    }
    float dot[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float a = 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u) a = fmaf(qf[g][u], kf[u], a);
      dot[g] = a;
    }
    // sums over the 16 lanes of the row (rotations by 8, 4, 2, 1): every lane gets them
#pragma unroll
    for (int g = 0; g < G; ++g) dot[g] += dpp_rot<0x128>(dot[g]);
#pragma unroll
    for (int g = 0; g < G; ++g) dot[g] += dpp_rot<0x124>(dot[g]);
#pragma unroll
    for (int g = 0; g < G; ++g) dot[g] += dpp_rot<0x122>(dot[g]);
#pragma unroll
    for (int g = 0; g < G; ++g) dot[g] += dpp_rot<0x121>(dot[g]);
    const int kl = kKeysPerPass * p + r;
    if (c < G) {
      float x = dot[0];
#pragma unroll
      for (int g = 1; g < G; ++g)
        if (c == g) x = dot[g];
      sX[c][kl] = key0 + kl < L ? x * sl2 : -__builtin_inff();
    }
  }
  __syncthreads();
  // logits out, one coalesced row per head
  float* tz = P.tz + (size_t)jt * G * L;
  for (int e = tid; e < G * kSlice; e += kTovaThreads) {
    const int g = e / kSlice, kl = e - g * kSlice;
    if (key0 + kl < L) tz[(size_t)g * L + key0 + kl] = sX[g][kl];
  }
  // per-head (max, sum) of the slice: wave wv takes heads wv, wv + 4, ...; two keys per lane
  for (int g = wv; g < G; g += kTovaThreads / 64) {
    const float x0 = sX[g][lane], x1 = sX[g][lane + 64];
    float m = fmaxf(x0, x1);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    float z = __builtin_amdgcn_exp2f(x0 - m) + __builtin_amdgcn_exp2f(x1 - m);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) z += __shfl_xor(z, o);
    if (lane == 0) {
      float* ts = P.tstat + (((size_t)jt * nsl + slice) * G + g) * 2;
      ts[0] = m;
      ts[1] = z;
    }
  }
}

template <int G>
__global__ __launch_bounds__(kTovaThreads) void tova_scores_kernel(const PrefillLaunch P) {
  __shared__ float sM[G], sRz[G];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int L = P.seq_len, nsl = P.n_slices;
  const int n_parts = (L + kTovaScoreKeys - 1) / kTovaScoreKeys;
  const int jt = blockIdx.x / n_parts, part = blockIdx.x - jt * n_parts;
  const int job = tova_job0(P) + jt;
  // fold each head's slice pairs: lanes stride over slices, then a butterfly over the wave
  for (int g = wv; g < G; g += kTovaThreads / 64) {
    float m = -__builtin_inff(), z = 0.f;
    for (int sl = lane; sl < nsl; sl += 64) {
      const float* ts = P.tstat + (((size_t)jt * nsl + sl) * G + g) * 2;
      if (z == 0.f) {
        m = ts[0];
        z = ts[1];
      } else {
        combine(m, z, ts[0], ts[1]);
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float m2 = __shfl_xor(m, o), z2 = __shfl_xor(z, o);
      if (z2 > 0.f) {
        if (z > 0.f) combine(m, z, m2, z2);
        else {
          m = m2;
          z = z2;
        }
      }
    }
    if (lane == 0) {
      sM[g] = m;
      sRz[g] = 1.f / z;   // z >= 1: the head's largest logit contributes exp2(0)
    }
  }
  __syncthreads();
  const float* tz = P.tz + (size_t)jt * G * L;
  float* S = P.S + (size_t)job * L;
  const float inv_g = 1.f / (float)G;
  const int j1 = min(L, (part + 1) * kTovaScoreKeys);
  for (int j = part * kTovaScoreKeys + tid; j < j1; j += kTovaThreads) {
    float a = 0.f;
#pragma unroll
    for (int g = 0; g < G; ++g) a += __builtin_amdgcn_exp2f(tz[(size_t)g * L + j] - sM[g]) * sRz[g];
    S[j] = a * inv_g;
  }
}

template <int G>
void launch_g(const PrefillLaunch& P, int n_jobs, hipStream_t st) {
  tova_logits_kernel<G><<<n_jobs * P.n_slices, kTovaThreads, 0, st>>>(P);
  const int n_parts = (P.seq_len + kTovaScoreKeys - 1) / kTovaScoreKeys;
  tova_scores_kernel<G><<<n_jobs * n_parts, kTovaThreads, 0, st>>>(P);
}

}  // namespace

int launch_tova(const PrefillLaunch& P, void* stream) {
  const int n_jobs = P.batch * (P.n_scored - P.n_window - P.n_full) * P.n_kv_heads;
  if (n_jobs <= 0) return 0;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  switch (P.group) {
    case 1: launch_g<1>(P, n_jobs, st); break;
    case 2: launch_g<2>(P, n_jobs, st); break;
    case 4: launch_g<4>(P, n_jobs, st); break;
    case 8: launch_g<8>(P, n_jobs, st); break;
    default: return (int)hipErrorInvalidValue;
  }
  return (int)hipGetLastError();
}

}  // namespace rkv
