// Decode-phase cache update for gfx950: one workgroup per (layer, sequence, KV head).
//
// H2O: the new key joins the C cached keys; every query head of the group scores the C+1
// entries (bf16 dot products accumulated in fp32), takes a softmax, and the group mean of the
// probabilities is added to each entry's fp32 accumulated score.  Among entries outside the
// protected recent window the smallest accumulated score (ties: smallest position) is
// evicted and the new token takes its slot.  TOVA: the same probabilities; an entry's score is
// their group mean at this step alone, every entry (the new one included) is a candidate, and
// the smallest score is evicted (ties: smallest position).  StreamingLLM: the oldest non-sink
// slot is replaced.  Keys are read with four lanes per 256-byte row (64 B per lane).
#include <hip/hip_runtime.h>

#include "rkv_internal.h"

namespace rkv {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / 64;

__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t v) { return __builtin_bit_cast(bf16x2, v); }

__device__ __forceinline__ float block_reduce_max(float v, float* sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  if (lane == 0) sh[wv] = v;
  __syncthreads();
  float r = sh[0];
#pragma unroll
  for (int i = 1; i < kDecWaves; ++i) r = fmaxf(r, sh[i]);
  __syncthreads();
  return r;
}

__device__ __forceinline__ float block_reduce_sum(float v, float* sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (lane == 0) sh[wv] = v;
  __syncthreads();
  float r = 0.f;
#pragma unroll
  for (int i = 0; i < kDecWaves; ++i) r += sh[i];
  __syncthreads();
  return r;
}

__device__ __forceinline__ uint64_t block_reduce_min_u64(uint64_t v, uint64_t* sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t y = __shfl_xor(v, o);
    v = y < v ? y : v;
  }
  if (lane == 0) sh[wv] = v;
  __syncthreads();
  uint64_t r = sh[0];
#pragma unroll
  for (int i = 1; i < kDecWaves; ++i) r = sh[i] < r ? sh[i] : r;
  __syncthreads();
  return r;
}

template <int G>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(const DecodeLaunch D) {
  extern __shared__ float sDyn[];
  __shared__ float shf[kDecWaves];
  __shared__ uint64_t shu[kDecWaves];
  const int tid = threadIdx.x;
  const int Hkv = D.n_kv_heads, B = D.batch;
  const int item = blockIdx.x;
  const int h = item % Hkv, s = (item / Hkv) % B, li = item / (Hkv * B);
  const DecodeLayer& ly = D.layer[li];
  const int C = ly.capacity;
  const int p = D.position;
  const size_t bh = (size_t)s * Hkv + h;
  int32_t* pos = ly.pos + bh * C;
  float* acc = ly.acc ? ly.acc + bh * C : nullptr;   // H2O layers only
  uint16_t* kc = ly.k_cache + bh * C * kHeadDim;
  uint16_t* vc = ly.v_cache + bh * C * kHeadDim;
  const uint16_t* knew = ly.k + bh * kHeadDim;
  const uint16_t* vnew = ly.v + bh * kHeadDim;

  uint64_t best = ~0ull;
  int victim = -1;
  if (ly.rule == RKV_STREAMING) {
    for (int e = tid; e < C; e += kDecThreads) {
      const int ps = pos[e];
      if (ps >= D.n_sink) {
        const uint64_t key = ((uint64_t)(uint32_t)ps << 32) | (uint32_t)e;
        best = key < best ? key : best;
      }
    }
    best = block_reduce_min_u64(best, shu);
    victim = best == ~0ull ? -1 : (int)(uint32_t)(best & 0xffffffffu);
  } else {
    float* sZ = sDyn;                      // [G][C+1] logits, then probabilities
    float* sAcc = sDyn + (size_t)G * (C + 1);  // [C+1] updated accumulated scores
    // query pairs for this lane's quarter of the head dimension
    const int qq = tid & 3;
    uint32_t qr[G][16];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint32_t* qp = reinterpret_cast<const uint32_t*>(ly.q + ((size_t)s * D.n_q_heads + h * G + g) * kHeadDim + 32 * qq);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(qp + 4 * i);
        qr[g][4 * i] = v[0]; qr[g][4 * i + 1] = v[1]; qr[g][4 * i + 2] = v[2]; qr[g][4 * i + 3] = v[3];
      }
    }
    for (int base = 0; base <= C; base += kDecThreads / 4) {
      const int e = base + (tid >> 2);
      float dot[G];
#pragma unroll
      for (int g = 0; g < G; ++g) dot[g] = 0.f;
      if (e <= C) {
        const uint16_t* kr = (e < C ? kc + (size_t)e * kHeadDim : knew) + 32 * qq;
        u32x4 kv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) kv[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kr + 8 * i));
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float d = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) d = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(kv[i][j]), as_bf16x2(qr[g][4 * i + j]), d, false);
          dot[g] = d;
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        dot[g] += __shfl_xor(dot[g], 1);
        dot[g] += __shfl_xor(dot[g], 2);
      }
      if (e <= C && qq == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) sZ[g * (C + 1) + e] = dot[g];
      }
    }
    __syncthreads();
    const float sl2 = D.scale_log2;
    for (int g = 0; g < G; ++g) {
      float m = -__builtin_inff();
      for (int e = tid; e <= C; e += kDecThreads) m = fmaxf(m, sZ[g * (C + 1) + e]);
      m = block_reduce_max(m, shf) * sl2;
      float sm = 0.f;
      for (int e = tid; e <= C; e += kDecThreads) {
        const float x = __builtin_amdgcn_exp2f(fmaf(sZ[g * (C + 1) + e], sl2, -m));
        sZ[g * (C + 1) + e] = x;
        sm += x;
      }
      sm = block_reduce_sum(sm, shf);
      const float inv = 1.0f / sm;
      for (int e = tid; e <= C; e += kDecThreads) sZ[g * (C + 1) + e] *= inv;
    }
    __syncthreads();
    // H2O: candidates have position <= p - r and the score accumulates; TOVA: every entry is a
    // candidate and the score is this step's alone
    const bool tova = ly.rule == RKV_TOVA;
    const int limit = tova ? p : p - ly.recent;
    for (int e = tid; e <= C; e += kDecThreads) {
      float pm = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) pm += sZ[g * (C + 1) + e];
      pm = pm / (float)G;
      const float a = (e < C && !tova ? acc[e] : 0.f) + pm;
      sAcc[e] = a;
      const int ps = e < C ? pos[e] : p;
      if (ps <= limit) {
        const uint64_t key = ((uint64_t)__float_as_uint(a) << 32) | (uint32_t)ps;
        best = key < best ? key : best;
      }
    }
    best = block_reduce_min_u64(best, shu);
    const int vpos = (int)(uint32_t)(best & 0xffffffffu);
    // slot holding the winning position (positions are distinct); C = the new token
    __shared__ int sVictim;
    if (tid == 0) sVictim = -1;
    __syncthreads();
    if (best != ~0ull) {
      for (int e = tid; e <= C; e += kDecThreads) {
        const int ps = e < C ? pos[e] : p;
        if (ps == vpos) sVictim = e;
      }
    }
    __syncthreads();
    victim = sVictim;
    if (victim == C) victim = -1;
    if (!tova)
      for (int e = tid; e < C; e += kDecThreads) acc[e] = (e == victim) ? sAcc[C] : sAcc[e];
  }
  // the new token takes the victim's slot
  if (victim >= 0) {
    if (tid < 16) {
      reinterpret_cast<u32x4*>(kc + (size_t)victim * kHeadDim)[tid] = reinterpret_cast<const u32x4*>(knew)[tid];
    } else if (tid < 32) {
      reinterpret_cast<u32x4*>(vc + (size_t)victim * kHeadDim)[tid - 16] = reinterpret_cast<const u32x4*>(vnew)[tid - 16];
    } else if (tid == 32) {
      pos[victim] = p;
    }
  }
  if (tid == 0 && ly.victim) ly.victim[bh] = victim;
}

}  // namespace

int launch_decode(const DecodeLaunch& D, int max_capacity, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const unsigned grid = (unsigned)(D.n_layers * D.batch * D.n_kv_heads);
  const size_t lds = sizeof(float) * (size_t)(D.group + 1) * (max_capacity + 1);
  static bool attr_set = false;
  if (!attr_set) {
    const void* fns[4] = {reinterpret_cast<const void*>(decode_kernel<1>), reinterpret_cast<const void*>(decode_kernel<2>),
                          reinterpret_cast<const void*>(decode_kernel<4>), reinterpret_cast<const void*>(decode_kernel<8>)};
    for (const void* f : fns) {
      hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 150 * 1024);
      if (e != hipSuccess) return (int)e;
    }
    attr_set = true;
  }
  profile_mark(kStageDecode, false, stream);
  switch (D.group) {
    case 1: decode_kernel<1><<<grid, kDecThreads, lds, st>>>(D); break;
    case 2: decode_kernel<2><<<grid, kDecThreads, lds, st>>>(D); break;
    case 4: decode_kernel<4><<<grid, kDecThreads, lds, st>>>(D); break;
    case 8: decode_kernel<8><<<grid, kDecThreads, lds, st>>>(D); break;
    default: return (int)hipErrorInvalidValue;
  }
  profile_mark(kStageDecode, true, stream);
  return (int)hipGetLastError();
}

}  // namespace rkv
