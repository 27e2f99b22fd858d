// Decode-phase cache update for gfx950: one workgroup per (layer, sequence, KV head).
//
// H2O: the new key joins the C cached keys; every query head of the group scores the C+1
// entries (bf16 dot products accumulated in fp32), takes a softmax, and the group mean of the
// probabilities is added to each entry's fp32 accumulated score.  Among entries outside the
// protected recent window the smallest accumulated score (ties: smallest position) is
// evicted and the new token takes its slot.  TOVA: the same probabilities; an entry's score is
// their group mean at this step alone, every entry (the new one included) is a candidate, and
// the smallest score is evicted (ties: smallest position).  StreamingLLM: the oldest non-sink
// slot is replaced.  Keys are read with 16 lanes per 256-byte row (16 bytes each), so one
// wave's load instruction reads four whole rows.
#include <hip/hip_runtime.h>

#include "rkv_internal.h"

namespace rkv {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / 64;

__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t v) { return __builtin_bit_cast(bf16x2, v); }

// Wave reductions by DPP: rotations inside each 16-lane row (every lane of a row ends with the
// row's value), then the four rows' values read from lanes 0, 16, 32 and 48 and combined in that
// order (a fixed order: the sums are reproducible).
template <int CTRL>
__device__ __forceinline__ float dppf(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}
template <int CTRL>
__device__ __forceinline__ uint32_t dppu(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xf, 0xf, false);
}
__device__ __forceinline__ float rows4(float v, int i) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16 * i));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dppf<0x128>(v));   // row_ror:8
  v = fmaxf(v, dppf<0x124>(v));   // row_ror:4
  v = fmaxf(v, dppf<0x122>(v));   // row_ror:2
  v = fmaxf(v, dppf<0x121>(v));   // row_ror:1
  return fmaxf(fmaxf(rows4(v, 0), rows4(v, 1)), fmaxf(rows4(v, 2), rows4(v, 3)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dppf<0x128>(v);
  v += dppf<0x124>(v);
  v += dppf<0x122>(v);
  v += dppf<0x121>(v);
  return (rows4(v, 0) + rows4(v, 1)) + (rows4(v, 2) + rows4(v, 3));
}
// minimum of a 64-bit key (compared as (high word, low word))
template <int CTRL>
__device__ __forceinline__ void min_step(uint32_t& hi, uint32_t& lo) {
  const uint32_t oh = dppu<CTRL>(hi), ol = dppu<CTRL>(lo);
  const bool take = oh < hi || (oh == hi && ol < lo);
  hi = take ? oh : hi;
  lo = take ? ol : lo;
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
  uint32_t hi = (uint32_t)(v >> 32), lo = (uint32_t)v;
  min_step<0x128>(hi, lo);
  min_step<0x124>(hi, lo);
  min_step<0x122>(hi, lo);
  min_step<0x121>(hi, lo);
  uint64_t r = ~0ull;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint64_t x = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)hi, 16 * i) << 32) |
                       (uint32_t)__builtin_amdgcn_readlane((int)lo, 16 * i);
    r = x < r ? x : r;
  }
  return r;
}

__device__ __forceinline__ uint64_t block_reduce_min_u64(uint64_t v, uint64_t* sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  v = wave_min_u64(v);
  if (lane == 0) sh[wv] = v;
  __syncthreads();
  uint64_t r = sh[0];
#pragma unroll
  for (int i = 1; i < kDecWaves; ++i) r = sh[i] < r ? sh[i] : r;
  __syncthreads();
  return r;
}

// Block-wide max / sum of G values at once (each value: its waves' results in wave order).
template <int G>
__device__ __forceinline__ void block_reduce_max_v(float (&v)[G], float* sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    v[g] = wave_max(v[g]);
    if (lane == 0) sh[wv * G + g] = v[g];
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float r = sh[g];
#pragma unroll
    for (int i = 1; i < kDecWaves; ++i) r = fmaxf(r, sh[i * G + g]);
    v[g] = r;
  }
  __syncthreads();
}
template <int G>
__device__ __forceinline__ void block_reduce_sum_v(float (&v)[G], float* sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    v[g] = wave_sum(v[g]);
    if (lane == 0) sh[wv * G + g] = v[g];
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float r = 0.f;
#pragma unroll
    for (int i = 0; i < kDecWaves; ++i) r += sh[i * G + g];
    v[g] = r;
  }
  __syncthreads();
}

template <int G>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(const DecodeLaunch D) {
  extern __shared__ float sDyn[];
  __shared__ float shf[kDecWaves * 8];
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
    // 16 lanes per entry: lane c (= tid % 16) takes the 16-byte chunk c of the head dimension, so
    // a wave's load instruction reads four whole 256-byte rows; lanes hold chunk c of every
    // query head.  An iteration covers 64 entries, entry base + tid / 16 + 16 j for j = 0..3.
    const int c16 = tid & 15, rsub = tid >> 4;
    u32x4 qr[G];
#pragma unroll
    for (int g = 0; g < G; ++g)
      qr[g] = reinterpret_cast<const u32x4*>(ly.q + ((size_t)s * D.n_q_heads + h * G + g) * kHeadDim)[c16];
    constexpr int kBlk = kDecThreads / 4;   // 64 entries per block
    // two blocks of key rows in flight: block b + 1's loads are outstanding while block b's dot
    // products run, and block b + 2's are issued right after them (two register sets,
    // alternating).  Every load is unconditional (entries past the end read the new token's row,
    // which the cache serves), so the compiler's waits leave the other block in flight.
    auto load_rows = [&](int base, u32x4 (&kv)[4]) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int e = base + rsub + 16 * j;
        const uint16_t* kr = e < C ? kc + (size_t)e * kHeadDim : knew;
        kv[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kr) + c16);
      }
    };
    float mx[G];
#pragma unroll
    for (int g = 0; g < G; ++g) mx[g] = -__builtin_inff();
    // dot products of the block at base (rows in kv), summed over the 16 lanes of each entry
    // (one DPP row, every lane gets the sum); one lane writes each logit to LDS
    auto process = [&](int base, const u32x4 (&kv)[4]) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int e = base + rsub + 16 * j;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float d = 0.f;
#pragma unroll
          for (int u = 0; u < 4; ++u) d = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(kv[j][u]), as_bf16x2(qr[g][u]), d, false);
          d += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, d), 0x128, 0xf, 0xf, false));
          d += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, d), 0x124, 0xf, 0xf, false));
          d += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, d), 0x122, 0xf, 0xf, false));
          d += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, d), 0x121, 0xf, 0xf, false));
          if (e <= C) {
            mx[g] = fmaxf(mx[g], d);
            if (c16 == ((j * G + g) & 15)) sZ[g * (C + 1) + e] = d;
          }
        }
      }
    };
    u32x4 ka[4], kb[4];
    load_rows(0, ka);
    load_rows(kBlk, kb);
    for (int base = 0; base <= C; base += 2 * kBlk) {
      process(base, ka);
      load_rows(base + 2 * kBlk, ka);
      process(base + kBlk, kb);
      load_rows(base + 3 * kBlk, kb);
    }
    // H2O: candidates have position <= p - r and the score accumulates; TOVA: every entry is a
    // candidate and the score is this step's alone
    const bool tova = ly.rule == RKV_TOVA;
    const int limit = tova ? p : p - ly.recent;
    // positions and accumulated scores of entries tid + 256 k (k < kDecPre), requested now so
    // that they arrive during the reductions and the exponential pass (the key registers are
    // free here); entries past those are read when visited
    constexpr int kDecPre = 4;
    int pre_pos[kDecPre];
    float pre_acc[kDecPre];
#pragma unroll
    for (int k = 0; k < kDecPre; ++k) {
      const int e = tid + kDecThreads * k;
      pre_pos[k] = e < C ? pos[e] : p;
      pre_acc[k] = e < C && !tova ? acc[e] : 0.f;
    }
    // every head's maximum and row sum in one pass over the logits, two block reductions
    const float sl2 = D.scale_log2;
    block_reduce_max_v<G>(mx, shf);   // its first barrier also publishes the logits in LDS
    float sm[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      mx[g] *= sl2;
      sm[g] = 0.f;
    }
    for (int e = tid; e <= C; e += kDecThreads) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float x = __builtin_amdgcn_exp2f(fmaf(sZ[g * (C + 1) + e], sl2, -mx[g]));
        sZ[g * (C + 1) + e] = x;
        sm[g] += x;
      }
    }
    block_reduce_sum_v<G>(sm, shf);
    float inv[G];
#pragma unroll
    for (int g = 0; g < G; ++g) inv[g] = 1.0f / sm[g];
    auto visit = [&](int e, float acc_e, int ps) {
      float pm = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) pm += sZ[g * (C + 1) + e] * inv[g];
      pm = pm / (float)G;
      const float a = acc_e + pm;
      sAcc[e] = a;
      if (ps <= limit) {
        const uint64_t key = ((uint64_t)__float_as_uint(a) << 32) | (uint32_t)ps;
        best = key < best ? key : best;
      }
    };
#pragma unroll
    for (int k = 0; k < kDecPre; ++k)
      if (tid + kDecThreads * k <= C) visit(tid + kDecThreads * k, pre_acc[k], pre_pos[k]);
    for (int e = tid + kDecThreads * kDecPre; e <= C; e += kDecThreads)
      visit(e, e < C && !tova ? acc[e] : 0.f, e < C ? pos[e] : p);
    best = block_reduce_min_u64(best, shu);
    const int vpos = (int)(uint32_t)(best & 0xffffffffu);
    // slot holding the winning position (positions are distinct); C = the new token
    __shared__ int sVictim;
    if (tid == 0) sVictim = -1;
    __syncthreads();
    if (best != ~0ull) {
#pragma unroll
      for (int k = 0; k < kDecPre; ++k)
        if (tid + kDecThreads * k <= C && pre_pos[k] == vpos) sVictim = tid + kDecThreads * k;
      for (int e = tid + kDecThreads * kDecPre; e <= C; e += kDecThreads) {
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
