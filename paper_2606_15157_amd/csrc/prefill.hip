// Prefill prompt compression kernels for gfx950 (CDNA4).
//
// One call runs, on the caller's stream:
//   zero_counters  clear the work-queue and barrier counters of the workspace
//   score_kernel   window Q K^T on bf16 MFMA (fp32 accumulate), causal mask, softmax
//                  normalised over all visible keys, window column sum, max-pool and
//                  query-group mean -> one fp32 score per (sequence, layer, KV head, key)
//   select_kernel  per (sequence, layer, KV head): top-k by (score desc, position asc)
//                  with a bitwise radix search for the k-th value and an ordered compaction
//   gather_kernel  copy the retained K and V rows (16 lanes x 16 B per 256-byte row)
//
// Softmax normalisation of a window row needs its maximum and sum over every key, while the
// window sum runs over rows.  A scoring work item owns 256 keys of one KV head for all of
// its G*w window rows and keeps its exponentials in registers; items publish per-row chunk
// maxima and sums, the last item of a head to arrive combines them, and every item then
// finishes its column sums with the head's normalisers.  Work items take tickets from an
// atomic counter, so the items of a head are always dispatched before any later ticket; a
// waiting item only ever waits for items that already hold tickets, which guarantees
// progress.  Each wait is bounded; on time-out the item flags the workspace status word.
//
// Cross-workgroup data is written and read with agent-scope relaxed atomics, which bypass the
// XCD-local caches; ordering uses workgroup fences plus vmcnt(0) waits, avoiding agent-scope
// fences (L2 flush and invalidate).
#include <hip/hip_runtime.h>

#include <math.h>

#include "rkv_internal.h"

namespace rkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kQStride = 136;            // bf16 per LDS row of Q: 128 + 8 padding (272 B)
constexpr int kTStride = 36;             // floats per row of a wave's 32x32 transpose tile
constexpr uint32_t kSpinLimit = 1u << 20;
constexpr int kSelectThreads = 512;
constexpr int kGatherThreads = 256;

__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __uint_as_float(__hip_atomic_load(reinterpret_cast<const uint32_t*>(p), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT));
}
// Wait until this wave's memory operations have completed (ordering only, no cache flush).
__device__ __forceinline__ void vmem_release() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8));
}
__device__ __forceinline__ void vmem_acquire() {
  __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8));
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__global__ void zero_counters(uint32_t* c, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) c[i] = 0u;
}

// ------------------------------------------------------------------------------------------
// Scoring.  NT = number of 32-row tiles of window rows per KV head (G * ceil(w/32), padded).
// Wave v of the work item computes the 32 x (NT*32) logit block of keys [c*256 + 32v, +32):
// MFMA A operand = 32 keys (straight from HBM into VGPRs), B operand = 32 query rows (LDS).
// Output element (key m, row n) of tile t lives in lane n + 32*((m/4)%2), register
// (m%4) + 4*(m/8): each lane owns one window row and 16 of the wave's keys.
// ------------------------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(kThreads) void score_kernel(const PrefillLaunch P) {
  constexpr int R = NT * 32;
  constexpr int kQBytes = R * kQStride * 2;
  constexpr int kTBytes = kWaves * 32 * kTStride * 4;
  constexpr int kUnion = kQBytes > kTBytes ? kQBytes : kTBytes;
  __shared__ __attribute__((aligned(16))) unsigned char sQT[kUnion];
  __shared__ float sRed[kWaves][R];
  __shared__ float sMax[R], sSum[R], sFac[R];
  __shared__ float sA[NT][kChunk];
  __shared__ int sTicket, sFlag;

  uint16_t* sQ = reinterpret_cast<uint16_t*>(sQT);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hf = lane >> 5, ln = lane & 31;
  uint32_t* counters = P.counters;

  if (tid == 0) sTicket = (int)atomicAdd(&counters[1], 1u);
  __syncthreads();
  const int ticket = sTicket;
  const int NC = P.n_chunks, L = P.seq_len, w = P.window, G = P.group, NTg = P.row_tiles_per_group;
  const int Hkv = P.n_kv_heads, B = P.batch;
  const int n_heads = B * P.n_scored * Hkv;
  const int hd = ticket / NC, c = ticket - hd * NC;
  const int h = hd % Hkv, s = (hd / Hkv) % B, slot = hd / (Hkv * B);
  const PrefillLayer& ly = P.layer[P.slot_layer[slot]];
  const int nt_used = G * NTg;

  // ---- window queries of this KV head's group -> LDS (zero rows for padding)
  {
    const uint16_t* qb = ly.q + (size_t)(s * P.n_q_heads + h * G) * w * kHeadDim;
    for (int e = tid; e < R * 16; e += kThreads) {
      const int row = e >> 4, piece = e & 15;
      const int g = row / (NTg * 32), i = row - g * (NTg * 32);
      u32x4 val = {0u, 0u, 0u, 0u};
      if (g < G && i < w) val = *reinterpret_cast<const u32x4*>(qb + (size_t)(g * w + i) * kHeadDim + piece * 8);
      *reinterpret_cast<u32x4*>(sQ + row * kQStride + piece * 8) = val;
    }
  }
  // ---- this wave's 32 keys, dims [64*hf, 64*hf + 64) per lane, straight to registers
  const int key0 = c * kChunk + wv * 32;
  const size_t head_base = (size_t)(s * Hkv + h) * L;
  u32x4 kf[8];
  {
    int key = key0 + ln;
    key = key < L ? key : L - 1;
    const uint16_t* kp = ly.k + (head_base + key) * kHeadDim + hf * 64;
#pragma unroll
    for (int st = 0; st < 8; ++st) kf[st] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kp + st * 8));
  }
  __syncthreads();

  f32x16 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
#pragma unroll
  for (int st = 0; st < 8; ++st) {
    const bf16x8 a = as_bf16x8(kf[st]);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t < nt_used) {
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(sQ + (t * 32 + ln) * kQStride + hf * 64 + st * 8);
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[t], 0, 0, 0);
      }
    }
  }

  // ---- mask (causal inside the window, ragged tail, padding rows) and chunk row maxima
  const float NEG_INF = -__builtin_inff();
  const bool need_mask = (key0 + 32 > L - w) || (nt_used < NT) || (w % 32 != 0);
  float part[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int row = t * 32 + ln;
    const int g = row / (NTg * 32), i = row - g * (NTg * 32);
    const bool rvalid = (t < nt_used) && (i < w);
    const int rpos = L - w + i;
    float m = NEG_INF;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float z = acc[t][r];
      if (need_mask) {
        const int kk = key0 + 8 * (r >> 2) + 4 * hf + (r & 3);
        if (!rvalid || kk >= L || kk > rpos) z = NEG_INF;
        acc[t][r] = z;
      }
      m = fmaxf(m, z);
    }
    m = fmaxf(m, __shfl_xor(m, 32));
    part[t] = m;
  }
  if (hf == 0) {
#pragma unroll
    for (int t = 0; t < NT; ++t) sRed[wv][t * 32 + ln] = part[t];
  }
  __syncthreads();
  if (tid < R) {
    float m = sRed[0][tid];
#pragma unroll
    for (int v = 1; v < kWaves; ++v) m = fmaxf(m, sRed[v][tid]);
    sMax[tid] = m;
  }
  __syncthreads();

  // ---- exponentials relative to the chunk maximum (kept in registers) and chunk row sums
  const float sl2 = P.scale_log2;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    float mref = sMax[t * 32 + ln];
    mref = (mref == NEG_INF) ? 0.f : mref * sl2;
    float sm = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e = __builtin_amdgcn_exp2f(fmaf(acc[t][r], sl2, -mref));
      acc[t][r] = e;
      sm += e;
    }
    sm += __shfl_xor(sm, 32);
    part[t] = sm;
  }
  if (hf == 0) {
#pragma unroll
    for (int t = 0; t < NT; ++t) sRed[wv][t * 32 + ln] = part[t];
  }
  __syncthreads();
  float* stat = P.stats + ((size_t)hd * NC + c) * R * 2;
  if (tid < R) {
    float sm = 0.f;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) sm += sRed[v][tid];
    sSum[tid] = sm;
    const float m = sMax[tid];
    store_coherent(stat + 2 * tid, m == NEG_INF ? NEG_INF : m * sl2);
    store_coherent(stat + 2 * tid + 1, sm);
  }
  vmem_release();
  __syncthreads();
  if (tid == 0) {
    const uint32_t old = __hip_atomic_fetch_add(&counters[2 + hd], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sFlag = (old == (uint32_t)(NC - 1)) ? 1 : 0;
  }
  __syncthreads();

  // ---- head normalisers: the last item combines every chunk's (max, sum), the others wait
  float* hstat = P.headstat + (size_t)hd * R * 2;
  if (sFlag) {
    vmem_acquire();
    if (tid < R) {
      float M = NEG_INF, S = 0.f;
      const float* st0 = P.stats + (size_t)hd * NC * R * 2 + 2 * tid;
      for (int cc = 0; cc < NC; ++cc) {
        const float m = load_coherent(st0 + (size_t)cc * R * 2);
        const float l = load_coherent(st0 + (size_t)cc * R * 2 + 1);
        if (l > 0.f) {
          if (m > M) { S = S * __builtin_amdgcn_exp2f(M - m) + l; M = m; }
          else S += l * __builtin_amdgcn_exp2f(m - M);
        }
      }
      const float inv = S > 0.f ? 1.0f / S : 0.f;
      store_coherent(hstat + 2 * tid, M);
      store_coherent(hstat + 2 * tid + 1, inv);
      sRed[0][tid] = M;
      sRed[1][tid] = inv;
    }
    vmem_release();
    __syncthreads();
    if (tid == 0) __hip_atomic_store(&counters[2 + n_heads + hd], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    if (tid == 0) {
      uint32_t it = 0;
      while (__hip_atomic_load(&counters[2 + n_heads + hd], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
        __builtin_amdgcn_s_sleep(2);
        if (++it > kSpinLimit) {
          atomicOr(&counters[0], 1u);
          break;
        }
      }
      vmem_acquire();
    }
    __syncthreads();
    if (tid < R) {
      sRed[0][tid] = load_coherent(hstat + 2 * tid);
      sRed[1][tid] = load_coherent(hstat + 2 * tid + 1);
    }
  }
  __syncthreads();
  if (tid < R) {
    const float mc = sMax[tid];
    const float M = sRed[0][tid], inv = sRed[1][tid];
    sFac[tid] = (inv == 0.f || mc == NEG_INF) ? 0.f : __builtin_amdgcn_exp2f(mc * sl2 - M) * inv;
  }
  __syncthreads();

  // ---- per query head column sums: scale by the row factor, transpose through LDS, reduce
  {
    float* T = reinterpret_cast<float*>(sQT) + wv * 32 * kTStride;
    for (int g = 0; g < G; ++g) {
      float v[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) v[r] = 0.f;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t >= g * NTg && t < (g + 1) * NTg) {
          const float f = sFac[t * 32 + ln];
#pragma unroll
          for (int r = 0; r < 16; ++r) v[r] = fmaf(f, acc[t][r], v[r]);
        }
      }
      // row ln, keys 8q + 4hf + {0..3}
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float4 x = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
        *reinterpret_cast<float4*>(T + ln * kTStride + 8 * q + 4 * hf) = x;
      }
      __builtin_amdgcn_wave_barrier();
      float sum = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) sum += T[(16 * hf + j) * kTStride + ln];
      sum += __shfl_xor(sum, 32);
      __builtin_amdgcn_wave_barrier();
      if (hf == 0) sA[g][wv * 32 + ln] = sum;
    }
  }
  __syncthreads();

  // ---- group mean (unpooled), in-chunk max-pool (SnapKV), scores and chunk-edge values
  const int cbase = c * kChunk;
  if (tid < kChunk) {
    const int key = cbase + tid;
    if (key < L) {
      float su = 0.f;
      for (int g = 0; g < G; ++g) su += sA[g][tid];
      su = su / (float)G;
      float* Srow = P.S + (size_t)hd * L;
      if (ly.rule == RKV_SNAPKV) {
        const int npre = L - w;
        float sc = su;
        if (key < npre) {
          const int ph = P.pool_half;
          const int lo = max(key - ph, cbase), hi = min(min(key + ph, cbase + kChunk - 1), npre - 1);
          sc = 0.f;
          for (int g = 0; g < G; ++g) {
            float m = NEG_INF;
            for (int t = lo; t <= hi; ++t) m = fmaxf(m, sA[g][t - cbase]);
            sc += m;
          }
          sc = sc / (float)G;
        }
        Srow[key] = sc;
        if (P.want_unpooled) P.Su[(size_t)hd * L + key] = su;
      } else {
        Srow[key] = su;
      }
    }
  }
  if (ly.rule == RKV_SNAPKV && P.pool_half > 0) {
    const int E = 4 * P.pool_half, twoP = 2 * P.pool_half;
    float* ed = P.edge + ((size_t)hd * NC + c) * G * E;
    for (int e = tid; e < G * E; e += kThreads) {
      const int g = e / E, o = e - g * E;
      const int kl = o < twoP ? o : kChunk - twoP + (o - twoP);
      ed[e] = (cbase + kl < L) ? sA[g][kl] : 0.f;
    }
  }
}

// ------------------------------------------------------------------------------------------
// Selection.  One workgroup per (layer slot, sequence, KV head).
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ int block_sum(int v, int* sh) {
  // sh: kSelectThreads / 64 + 1 ints
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (lane == 0) sh[wv] = v;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int i = 0; i < kSelectThreads / 64; ++i) t += sh[i];
  __syncthreads();
  return t;
}

// exclusive prefix over threads of a per-thread count; returns the prefix, *total gets the sum
__device__ __forceinline__ int block_exclusive_scan(int v, int* sh, int* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o);
    if (lane >= o) inc += y;
  }
  if (lane == 63) sh[wv] = inc;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSelectThreads / 64; ++i) {
    const int x = sh[i];
    before += (i < wv) ? x : 0;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return before + inc - v;
}

__global__ __launch_bounds__(kSelectThreads) void select_kernel(const PrefillLaunch P) {
  extern __shared__ float sS[];
  __shared__ int sh[kSelectThreads / 64 + 1];
  const int tid = threadIdx.x;
  const int hd = blockIdx.x;
  const int Hkv = P.n_kv_heads, B = P.batch, L = P.seq_len, w = P.window, G = P.group, NC = P.n_chunks;
  const int h = hd % Hkv, s = (hd / Hkv) % B, slot = hd / (Hkv * B);
  const PrefillLayer& ly = P.layer[P.slot_layer[slot]];
  const int bh = s * Hkv + h;
  const float* Srow = P.S + (size_t)hd * L;
  const bool snap = ly.rule == RKV_SNAPKV;
  // candidate range over which scores are defined
  const int n_score = ly.all ? (snap ? L - w : L) : ly.cand_end;

  for (int j = tid; j < n_score; j += kSelectThreads) sS[j] = Srow[j];
  __syncthreads();
  // SnapKV: redo the pooled score of positions within pool_half of an interior chunk boundary
  if (snap && P.pool_half > 0 && n_score > 0) {
    const int ph = P.pool_half, E = 4 * ph, twoP = 2 * ph;
    const float NEG_INF = -__builtin_inff();
    const int npre = L - w;
    for (int e = tid; e < (NC - 1) * twoP; e += kSelectThreads) {
      const int cb = 1 + e / twoP, o = e - (e / twoP) * twoP;
      const int bnd = cb * kChunk;
      const int j = bnd - ph + o;
      if (j < 0 || j >= npre || j >= n_score) continue;
      const float* left = P.edge + ((size_t)hd * NC + (cb - 1)) * G * E;   // keys [bnd-2P, bnd) at [2P, 4P)
      const float* right = P.edge + ((size_t)hd * NC + cb) * G * E;        // keys [bnd, bnd+2P) at [0, 2P)
      const int lo = max(j - ph, 0), hi = min(j + ph, npre - 1);
      float sc = 0.f;
      for (int g = 0; g < G; ++g) {
        float m = NEG_INF;
        for (int t = lo; t <= hi; ++t) {
          const float a = (t < bnd) ? left[g * E + twoP + (t - (bnd - twoP))] : right[g * E + (t - bnd)];
          m = fmaxf(m, a);
        }
        sc += m;
      }
      sS[j] = sc / (float)G;
    }
    __syncthreads();
  }
  if (ly.score) {
    float* so = ly.score + (size_t)bh * L;
    for (int j = tid; j < n_score; j += kSelectThreads) so[j] = sS[j];
  }

  int32_t* idx = ly.idx + (size_t)bh * ly.n_keep;
  float* acc = ly.acc ? ly.acc + (size_t)bh * ly.n_keep : nullptr;
  const float* accsrc = snap ? P.Su + (size_t)hd * L : Srow;
  if (ly.all) {
    for (int m = tid; m < ly.n_keep; m += kSelectThreads) {
      idx[m] = m;
      if (acc) acc[m] = accsrc[m];
    }
    return;
  }
  const int n = ly.cand_end, k = ly.k_sel;
  if (k > 0) {
    // k-th largest candidate score: largest pattern T with #(x >= T) >= k (scores are >= 0,
    // so unsigned order of the bit patterns is the numeric order)
    uint32_t prefix = 0u;
    for (int bit = 30; bit >= 0; --bit) {
      const uint32_t cand = prefix | (1u << bit);
      int cnt = 0;
      for (int j = tid; j < n; j += kSelectThreads) cnt += (__float_as_uint(sS[j]) >= cand) ? 1 : 0;
      cnt = block_sum(cnt, sh);
      if (cnt >= k) prefix = cand;
    }
    const uint32_t tau = prefix;
    // ordered compaction over contiguous per-thread segments
    const int seg = (n + kSelectThreads - 1) / kSelectThreads;
    const int j0 = min(n, tid * seg), j1 = min(n, j0 + seg);
    int gt = 0, eq = 0;
    for (int j = j0; j < j1; ++j) {
      const uint32_t x = __float_as_uint(sS[j]);
      gt += x > tau;
      eq += x == tau;
    }
    int tot_gt, tot_eq;
    const int pre_gt = block_exclusive_scan(gt, sh, &tot_gt);
    const int pre_eq = block_exclusive_scan(eq, sh, &tot_eq);
    const int need = k - tot_gt;   // ties at tau taken in position order
    int out = pre_gt + min(pre_eq, need);
    int er = pre_eq;
    for (int j = j0; j < j1; ++j) {
      const uint32_t x = __float_as_uint(sS[j]);
      bool take = x > tau;
      if (x == tau) {
        take = er < need;
        ++er;
      }
      if (take) {
        idx[out] = j;
        if (acc) acc[out] = accsrc[j];
        ++out;
      }
    }
  }
  const int nf = ly.forced_hi - ly.forced_lo;
  for (int t = tid; t < nf; t += kSelectThreads) {
    idx[k + t] = ly.forced_lo + t;
    if (acc) acc[k + t] = accsrc[ly.forced_lo + t];
  }
}

// ------------------------------------------------------------------------------------------
// Gather: 16 consecutive threads copy one 256-byte row of K and of V.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kGatherThreads) void gather_kernel(const PrefillLaunch P) {
  const int64_t gid = (int64_t)blockIdx.x * kGatherThreads + threadIdx.x;
  const int64_t row = gid >> 4;
  const int piece = (int)(gid & 15);
  if (row >= P.rows_prefix[P.n_layers]) return;
  int li = 0;
  while (li + 1 < P.n_layers && P.rows_prefix[li + 1] <= row) ++li;
  const PrefillLayer& ly = P.layer[li];
  const int64_t local = row - P.rows_prefix[li];
  const int n_keep = ly.n_keep;
  const int64_t bh = local / n_keep;
  const int m = (int)(local - bh * n_keep);
  int pos;
  if (ly.slot >= 0) {
    pos = ly.idx[bh * n_keep + m];
  } else {
    pos = ly.all ? m : (m < ly.cand_end ? m : ly.forced_lo + (m - ly.cand_end));
    if (piece == 0) {
      ly.idx[bh * n_keep + m] = pos;
      if (ly.acc) ly.acc[bh * n_keep + m] = 0.f;
    }
  }
  const int L = P.seq_len;
  const size_t src = ((size_t)bh * L + pos) * kHeadDim + piece * 8;
  const size_t dst = ((size_t)bh * n_keep + m) * kHeadDim + piece * 8;
  const u32x4 kv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ly.k + src));
  const u32x4 vv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ly.v + src));
  *reinterpret_cast<u32x4*>(ly.k_out + dst) = kv;
  *reinterpret_cast<u32x4*>(ly.v_out + dst) = vv;
}

}  // namespace

int launch_prefill(const PrefillLaunch& P, int row_tiles, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int n_heads = P.batch * P.n_scored * P.n_kv_heads;
  if (P.n_scored > 0) {
    const int nc = 2 + 2 * n_heads;
    profile_mark(kStageZero, false, stream);
    zero_counters<<<(nc + 255) / 256, 256, 0, st>>>(P.counters, nc);
    profile_mark(kStageZero, true, stream);
    const unsigned grid = (unsigned)n_heads * (unsigned)P.n_chunks;
    profile_mark(kStageScore, false, stream);
    if (row_tiles == 4) score_kernel<4><<<grid, kThreads, 0, st>>>(P);
    else score_kernel<8><<<grid, kThreads, 0, st>>>(P);
    profile_mark(kStageScore, true, stream);
    const size_t lds = sizeof(float) * (size_t)P.seq_len;
    static bool attr_set = false;
    if (!attr_set) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(select_kernel),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, 150 * 1024);
      if (e != hipSuccess) return (int)e;
      attr_set = true;
    }
    profile_mark(kStageSelect, false, stream);
    select_kernel<<<n_heads, kSelectThreads, lds, st>>>(P);
    profile_mark(kStageSelect, true, stream);
  }
  const int64_t rows = P.rows_prefix[P.n_layers];
  if (rows > 0) {
    const int64_t threads = rows * 16;
    const unsigned grid = (unsigned)((threads + kGatherThreads - 1) / kGatherThreads);
    profile_mark(kStageGather, false, stream);
    gather_kernel<<<grid, kGatherThreads, 0, st>>>(P);
    profile_mark(kStageGather, true, stream);
  }
  return (int)hipGetLastError();
}

}  // namespace rkv
