// Prefill prompt compression for gfx950 (CDNA4): one fused kernel per launch group.
//
// Per (sequence, scored layer, KV head) -- a "head" -- the window scores are
//   A[g][j] = sum_i softmax_j(Q[g,i] . K[j] / sqrt(d))      (w window rows per query head g)
//   S[j]    = mean_g maxpool(A[g])[j]  (SnapKV)  or  mean_g A[g][j]  (H2O)
// The softmax of a window row is normalised over every key while the window sum runs over
// rows, so a head is done in two passes over its keys, each split into 512-key chunks:
//   stats item  (head, chunk): logits on MFMA (K chunk as the 32-row A operand, window queries
//               from LDS as B), per-row running max and sum of exponentials; the last chunk of
//               the head to finish folds all chunks into one log-normaliser per row;
//   score item  (head, chunk): the same logits again (the chunk's K is re-read from the
//               on-die caches: score items run a fixed number of steps after their head's stats
//               items), probabilities exp2(z - normaliser), column sums per query head inside
//               each lane (queries as the A operand put a key in every lane), max-pool inside
//               the chunk, group mean -> S;
//   select item (head): fixes the pooled score next to chunk borders, finds the k-th largest
//               score with three radix-histogram passes, writes the retained positions in
//               ascending order (ties at the k-th value taken by position);
//   gather item (head, part): copies the retained K and V rows, 16 lanes x 16 B per row.
// Layers that need no scores (StreamingLLM, Full, or budgets covering the prompt) get copy
// items only.  Items take tickets from an atomic counter, so they start in ticket order; an item
// waits only for items with earlier tickets (which never wait for later ones), and every wait is
// bounded (on time-out the workspace status word is set and the item carries on).
//
// Data handed between workgroups goes through agent-scope relaxed atomics (they bypass the
// XCD-local caches); ordering uses workgroup fences plus vmcnt(0) waits rather than agent-scope
// fences, which would flush and invalidate L2.
#include <hip/hip_runtime.h>

#include <math.h>

#include <algorithm>

#include "rkv_internal.h"

namespace rkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;            // 4 waves, one per SIMD
constexpr int kWaves = kThreads / 64;
constexpr int kKeysPerWave = kChunk / kWaves;   // 128 keys = 4 tiles of 32
constexpr int kTilesPerWave = kKeysPerWave / 32;
constexpr int kKDepth = 2;               // key tiles in registers per wave (1 loading ahead)
static_assert(kTilesPerWave % kKDepth == 0, "tile loop is unrolled by the ring depth");
constexpr int kRowTilesPerPass = 1;      // row tiles whose accumulators are live at once
constexpr int kQStride = 136;            // bf16 per LDS row of Q: 128 + 8 padding (272 B)
constexpr uint32_t kSpinLimit = 1u << 21;
constexpr int kHistBins = 2048;

enum ItemType { kItemStats = 0, kItemScore = 1, kItemSelect = 2, kItemGather = 3, kItemCopy = 4 };

__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __float_as_uint(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_coherent(int32_t* p, int32_t v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), (uint32_t)v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __uint_as_float(__hip_atomic_load(reinterpret_cast<const uint32_t*>(p), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ int32_t load_coherent(const int32_t* p) {
  return (int32_t)__hip_atomic_load(reinterpret_cast<const uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_coherent2(float* p, float a, float b) {
  const uint64_t v = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_coherent2(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
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
// Bounded wait (one thread) until *flag >= target.
__device__ __forceinline__ void wait_at_least(uint32_t* flag, uint32_t target, uint32_t* status) {
  uint32_t it = 0;
  while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
    __builtin_amdgcn_s_sleep(2);
    if (++it > kSpinLimit) {
      atomicOr(status, 1u);
      break;
    }
  }
  vmem_acquire();
}

// Online combination of (max, sum) pairs in log2 units.
__device__ __forceinline__ void combine_ms(float& M, float& S, float m, float l) {
  if (!(l > 0.f)) return;
  if (m > M) {
    S = S * __builtin_amdgcn_exp2f(M - m) + l;
    M = m;
  } else {
    S += l * __builtin_amdgcn_exp2f(m - M);
  }
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Clears the counters and fills the statistics, score and chunk-edge regions with the NaN
// pattern that marks "not written yet" (every written value is a number).
__global__ void reset_workspace(uint32_t* counters, int n_counters, u32x4* fill, int64_t n_fill) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = i0; i < n_counters; i += stride) counters[i] = 0u;
  const u32x4 nan4 = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};
  for (int64_t i = i0; i < n_fill; i += stride) fill[i] = nan4;
}

__device__ __forceinline__ bool unwritten(float x) { return x != x; }

// ---------------------------------------------------------------------------------------------
// Work-item decoding.
// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ int64_t clampi(int64_t x, int64_t lo, int64_t hi) { return x < lo ? lo : (x > hi ? hi : x); }

// Tickets issued before step s.  Step s holds the stats items of head s, the score items of
// head s - lb, the select item of head s - lb - ls and the gather items of head s - lb - ls - lg.
struct Lags {
  int64_t b, s, g;
};
__device__ __forceinline__ int64_t step_prefix(int64_t s, int64_t nH, int64_t NC, const Lags& lag) {
  return NC * clampi(s, 0, nH) + NC * clampi(s - lag.b, 0, nH) + clampi(s - lag.b - lag.s, 0, nH) +
         (int64_t)kGatherParts * clampi(s - lag.b - lag.s - lag.g, 0, nH);
}

struct Item {
  int type, head, chunk, part;
};

__device__ Item decode_item(int64_t t, const PrefillLaunch& P, int nH) {
  Item it{};
  const int64_t NC = P.n_chunks;
  const Lags lag{P.lag_score, P.lag_select, P.lag_gather};
  const int64_t n_steps = nH + lag.b + lag.s + lag.g;
  const int64_t scored_total = nH > 0 ? step_prefix(n_steps, nH, NC, lag) : 0;
  if (t >= scored_total) {
    const int64_t u = t - scored_total;
    it.type = kItemCopy;
    it.part = (int)(u % kGatherParts);
    it.head = (int)(u / kGatherParts);   // (unscored layer, sequence, KV head)
    return it;
  }
  int64_t lo = 0, hi = n_steps - 1;      // largest s with prefix(s) <= t
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (step_prefix(mid, nH, NC, lag) <= t) lo = mid; else hi = mid - 1;
  }
  const int64_t s = lo;
  int64_t w = t - step_prefix(s, nH, NC, lag);
  if (s < nH) {
    if (w < NC) { it.type = kItemStats; it.head = (int)s; it.chunk = (int)w; return it; }
    w -= NC;
  }
  const int64_t hb = s - lag.b, hs = hb - lag.s, hg = hs - lag.g;
  if (hb >= 0 && hb < nH) {
    if (w < NC) { it.type = kItemScore; it.head = (int)hb; it.chunk = (int)w; return it; }
    w -= NC;
  }
  if (hs >= 0 && hs < nH) {
    if (w < 1) { it.type = kItemSelect; it.head = (int)hs; return it; }
    w -= 1;
  }
  it.type = kItemGather;
  it.head = (int)hg;
  it.part = (int)w;
  return it;
}

// ---------------------------------------------------------------------------------------------
// Shared pieces of the stats and score items.
// ---------------------------------------------------------------------------------------------
template <int NT, int NTG>
__device__ __forceinline__ void load_q_to_lds(uint16_t* sQ, const PrefillLaunch& P, const PrefillLayer& ly, int s, int h) {
  constexpr int R = NT * 32;
  constexpr int kPer = R * 16 / kThreads;   // 16-byte pieces per thread
  const int G = P.group, w = P.window;
  const uint16_t* qb = ly.q + (size_t)(s * P.n_q_heads + h * G) * w * kHeadDim;
  u32x4 val[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {       // all loads in flight together
    const int e = threadIdx.x + i * kThreads;
    const int row = e >> 4, piece = e & 15;
    const int t = row >> 5;
    const int g = t / NTG, ii = (t - g * NTG) * 32 + (row & 31);
    val[i] = u32x4{0u, 0u, 0u, 0u};
    if (g < G && ii < w) val[i] = *reinterpret_cast<const u32x4*>(qb + (size_t)(g * w + ii) * kHeadDim + piece * 8);
  }
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int e = threadIdx.x + i * kThreads;
    *reinterpret_cast<u32x4*>(sQ + (e >> 4) * kQStride + (e & 15) * 8) = val[i];
  }
}

// Lane of a 32-key tile: key `key` (clamped into the head), dims 64*hf + [0, 64).
__device__ __forceinline__ void load_k_frag(u32x4 (&kf)[8], const uint16_t* khead, int key, int L, int hf) {
  key = key < L ? key : L - 1;
  const uint16_t* kp = khead + (size_t)key * kHeadDim + hf * 64;
#pragma unroll
  for (int st = 0; st < 8; ++st) kf[st] = *reinterpret_cast<const u32x4*>(kp + st * 8);
}

// One 32-key tile against NH row tiles starting at t0: 8 k-steps of 16 dims.  KEYS_AS_COLUMNS = false puts
// the keys on the MFMA A operand (output lane = window row), true puts the window queries on A
// (output lane = key).  The scheduling barriers keep the compiler from hoisting all 32 query
// fragment reads from LDS ahead of the MFMAs (that costs 128 VGPRs).
template <int NH, bool KEYS_AS_COLUMNS>
__device__ __forceinline__ void mfma_tile(f32x16 (&acc)[NH], const u32x4 (&kf)[8], const uint16_t* sQ, int ln, int hf,
                                          int t0, int nt_used) {
#pragma unroll
  for (int i = 0; i < NH; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
#pragma unroll
  for (int st = 0; st < 8; ++st) {
    const bf16x8 kb = as_bf16x8(kf[st]);
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      if (t0 + i < nt_used) {
        const bf16x8 qf = *reinterpret_cast<const bf16x8*>(sQ + ((t0 + i) * 32 + ln) * kQStride + hf * 64 + st * 8);
        if (KEYS_AS_COLUMNS) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf, kb, acc[i], 0, 0, 0);
        else acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb, qf, acc[i], 0, 0, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Masking of one accumulator tile (causal inside the window, ragged tail, padding rows).
template <int NTG>
__device__ __forceinline__ void mask_rows_lane(f32x16& acc, int t, int ln, int hf, int tile_key0, int G, int w, int L) {
  // lane = window row ln of tile t, registers = keys tile_key0 + 8(r/4) + 4hf + r%4
  const int g = t / NTG, i = (t - g * NTG) * 32 + ln;
  const bool valid = g < G && i < w;
  const int last = min(L - 1, L - w + i);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int kk = tile_key0 + 8 * (r >> 2) + 4 * hf + (r & 3);
    if (!valid || kk > last) acc[r] = -__builtin_inff();
  }
}
template <int NTG>
__device__ __forceinline__ void mask_rows_regs(f32x16& p, int t, int hf, int key, int G, int w, int L) {
  // lane = key, registers = window rows t*32 + 8(r/4) + 4hf + r%4
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int rr = 8 * (r >> 2) + 4 * hf + (r & 3);
    const int g = t / NTG, i = (t - g * NTG) * 32 + rr;
    if (!(g < G && i < w && key < L && key <= L - w + i)) p[r] = 0.f;
  }
}

// Window-row bookkeeping for row tile t, row-in-tile rr: whether the row exists and its position.
template <int NTG>
__device__ __forceinline__ bool row_visible(int t, int rr, int key, int G, int w, int L) {
  const int g = t / NTG, i = (t - g * NTG) * 32 + rr;
  return g < G && i < w && key < L && key <= L - w + i;
}

// ---------------------------------------------------------------------------------------------
// The fused kernel.  NT = row tiles (G * NTG, padded), NTG = row tiles per query head.
// ---------------------------------------------------------------------------------------------
template <int NT, int NTG>
__global__ __launch_bounds__(kThreads, 2) void evict_kernel(const PrefillLaunch P) {
  constexpr int R = NT * 32;
  constexpr int NG = NT / NTG;           // query heads per KV head supported by this instance
  constexpr int kQBytes = R * kQStride * 2;
  constexpr int kAuxA = kWaves * R * 2 * 4;
  constexpr int kGroupsB = kThreads / R > 0 ? kThreads / R : 1;
  constexpr int kAuxB = (NG * kChunk + R + kGroupsB * R * 2) * 4;
  constexpr int kAuxBytes = kAuxA > kAuxB ? kAuxA : kAuxB;
  constexpr int kItemBytes = kQBytes + kAuxBytes;
  constexpr int kSelFixed = kHistBins * 4 + 64;
  constexpr int kLdsBytes = kItemBytes > kSelFixed + 4096 ? kItemBytes : kSelFixed + 4096;
  __shared__ __attribute__((aligned(16))) unsigned char smem[kLdsBytes];
  __shared__ int sInfo[4];

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hf = lane >> 5, ln = lane & 31;
  uint32_t* counters = P.counters;
  uint32_t* status = counters;
  const int Hkv = P.n_kv_heads, B = P.batch, L = P.seq_len, w = P.window, G = P.group, NC = P.n_chunks;
  const int nH = B * P.n_scored * Hkv;
  uint32_t* selDone = counters + 2;

  if (tid == 0) {
    // Workgroups are dispatched in index order (round-robin over the XCDs), so the block index
    // is the ticket: every item an item waits for has a smaller index and has been dispatched.
    const Item it = decode_item((int64_t)blockIdx.x, P, nH);
    sInfo[0] = it.type; sInfo[1] = it.head; sInfo[2] = it.chunk; sInfo[3] = it.part;
  }
  __syncthreads();
  const int type = sInfo[0], head = sInfo[1], chunk = sInfo[2], part = sInfo[3];
  const float sl2 = P.scale_log2;
  const float NEG_INF = -__builtin_inff();

  // ============================================================== gather / copy items
  if (type == kItemGather || type == kItemCopy) {
    const int h = head % Hkv, s = (head / Hkv) % B, li = head / (Hkv * B);
    const PrefillLayer& ly = P.layer[type == kItemGather ? P.slot_layer[li] : P.unscored_layer[li]];
    const int bh = s * Hkv + h;
    const int n_keep = ly.n_keep;
    const int r0 = (int)((int64_t)part * n_keep / kGatherParts), r1 = (int)((int64_t)(part + 1) * n_keep / kGatherParts);
    if (r1 <= r0) return;
    if (type == kItemGather) {
      if (tid == 0) wait_at_least(&selDone[head], 1u, status);
      __syncthreads();
    }
    int32_t* idx = ly.idx + (size_t)bh * n_keep;
    const size_t hbase = (size_t)bh * L;
    const int piece = tid & 15, rsub = tid >> 4;
    constexpr int kRowsPerPass = (kThreads / 16) * 8;   // 16 row groups x 8 rows in flight
    for (int m0 = r0; m0 < r1; m0 += kRowsPerPass) {
      int pos[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int m = m0 + rsub + 16 * u;
        pos[u] = -1;
        if (m < r1) {
          if (type == kItemGather) pos[u] = load_coherent(idx + m);
          else pos[u] = ly.all ? m : (m < ly.cand_end ? m : ly.forced_lo + (m - ly.cand_end));
        }
      }
      u32x4 kv[8], vv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (pos[u] >= 0) {
          const size_t src = (hbase + pos[u]) * kHeadDim + piece * 8;
          kv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ly.k + src));
          vv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ly.v + src));
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int m = m0 + rsub + 16 * u;
        if (pos[u] >= 0) {
          const size_t dst = ((size_t)bh * n_keep + m) * kHeadDim + piece * 8;
          __builtin_nontemporal_store(kv[u], reinterpret_cast<u32x4*>(ly.k_out + dst));
          __builtin_nontemporal_store(vv[u], reinterpret_cast<u32x4*>(ly.v_out + dst));
          if (type == kItemCopy && piece == 0) {
            idx[m] = pos[u];
            if (ly.acc) ly.acc[(size_t)bh * n_keep + m] = 0.f;
          }
        }
      }
    }
    return;
  }

  const int h = head % Hkv, s = (head / Hkv) % B, slot = head / (Hkv * B);
  const PrefillLayer& ly = P.layer[P.slot_layer[slot]];
  const int bh = s * Hkv + h;
  const bool snap = ly.rule == RKV_SNAPKV;

  // ============================================================== select item
  if (type == kItemSelect) {
    int* sHist = reinterpret_cast<int*>(smem);
    int* sScan = sHist + kHistBins;          // kWaves ints
    int* sSel = sScan + 8;                   // 2 ints
    float* sCache = reinterpret_cast<float*>(smem + kSelFixed);
    const int cache_cap = (kLdsBytes - kSelFixed) / 4;
    float* Srow = P.S + (size_t)head * L;
    const int n_score = ly.all ? (snap ? L - w : L) : ly.cand_end;
    const int ph = P.pool_half, E = 4 * ph, twoP = 2 * ph;
    const bool fix = snap && ph > 0 && n_score > 0 && NC > 1;
    const int n_edge = fix ? NC * G * E : 0;
    const bool cached = n_score + n_edge <= cache_cap;
    float* sEdge = sCache + n_score;          // chunk-edge column sums (cached path)
    const float* Erow = P.edge + (size_t)head * NC * G * E;
    // wait (bounded) until every score of the head is written (and the unpooled scores when they
    // seed acc_out); keep the candidate scores and the chunk-edge values in LDS when they fit
    const float* Surow = P.Su + (size_t)head * L;
    const bool need_su = snap && ly.acc != nullptr;
    for (int j0 = tid; j0 < L; j0 += kThreads * 8) {
      float x[8], y[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kThreads;
        x[u] = j < L ? load_coherent(Srow + j) : 0.f;
        y[u] = (need_su && j < L) ? load_coherent(Surow + j) : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kThreads;
        uint32_t it = 0;
        while (unwritten(x[u]) || unwritten(y[u])) {
          __builtin_amdgcn_s_sleep(2);
          x[u] = load_coherent(Srow + j);
          if (need_su) y[u] = load_coherent(Surow + j);
          if (++it > kSpinLimit) {
            atomicOr(status, 1u);
            x[u] = 0.f;
            y[u] = 0.f;
          }
        }
        if (cached && j < n_score) sCache[j] = x[u];
      }
    }
    auto edge_at = [&](int e) -> float {
      float a = load_coherent(Erow + e);
      uint32_t it = 0;
      while (unwritten(a)) {
        __builtin_amdgcn_s_sleep(2);
        a = load_coherent(Erow + e);
        if (++it > kSpinLimit) {
          atomicOr(status, 1u);
          a = 0.f;
        }
      }
      return a;
    };
    if (fix && cached) {
      for (int e0 = tid; e0 < n_edge; e0 += kThreads * 4) {
        float a[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) a[u] = e0 + u * kThreads < n_edge ? load_coherent(Erow + e0 + u * kThreads) : 0.f;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = e0 + u * kThreads;
          if (e < n_edge) sEdge[e] = unwritten(a[u]) ? edge_at(e) : a[u];
        }
      }
    }
    __syncthreads();
    // SnapKV: redo the pooled score of positions within pool_half of an interior chunk border
    if (fix) {
      const int npre = L - w;
      for (int e = tid; e < (NC - 1) * twoP; e += kThreads) {
        const int cb = 1 + e / twoP, o = e - (e / twoP) * twoP;
        const int bnd = cb * kChunk;
        const int j = bnd - ph + o;
        if (j < 0 || j >= npre || j >= n_score) continue;
        // chunk cb-1 holds keys [bnd-2P, bnd) at offsets [2P, 4P); chunk cb keys [bnd, bnd+2P) at [0, 2P)
        const int left = (cb - 1) * G * E, right = cb * G * E;
        const int lo = max(j - ph, 0), hi = min(j + ph, npre - 1);
        float sc = 0.f;
        for (int g = 0; g < G; ++g) {
          float m = NEG_INF;
          for (int t = lo; t <= hi; ++t) {
            const int ei = (t < bnd) ? left + g * E + twoP + (t - (bnd - twoP)) : right + g * E + (t - bnd);
            m = fmaxf(m, cached ? sEdge[ei] : edge_at(ei));
          }
          sc += m;
        }
        if (cached) sCache[j] = sc / (float)G;
        else store_coherent(Srow + j, sc / (float)G);
      }
      if (!cached) vmem_release();
    }
    __syncthreads();
    auto get = [&](int j) -> float { return cached ? sCache[j] : load_coherent(Srow + j); };
    if (ly.score) {
      float* so = ly.score + (size_t)bh * L;
      for (int j = tid; j < n_score; j += kThreads) so[j] = get(j);
    }
    int32_t* idx = ly.idx + (size_t)bh * ly.n_keep;
    float* acc = ly.acc ? ly.acc + (size_t)bh * ly.n_keep : nullptr;
    const float* accsrc = snap ? Surow : Srow;
    if (ly.all) {
      for (int m = tid; m < ly.n_keep; m += kThreads) store_coherent(idx + m, m);
    } else {
      const int n = ly.cand_end, k = ly.k_sel;
      if (k > 0) {
        // k-th largest candidate score: three radix passes over the 31 value bits (scores are
        // >= 0, so the unsigned order of their bit patterns is the numeric order)
        uint32_t prefix = 0u, pmask = 0u;
        int kk = k;
#pragma unroll 1
        for (int pass = 0; pass < 3; ++pass) {
          const int shift = pass == 0 ? 20 : (pass == 1 ? 10 : 0);
          const int nb = pass == 0 ? 2048 : 1024;
          for (int b = tid; b < nb; b += kThreads) sHist[b] = 0;
          __syncthreads();
          for (int j = tid; j < n; j += kThreads) {
            const uint32_t x = __float_as_uint(get(j));
            if ((x & pmask) == prefix) atomicAdd(&sHist[(x >> shift) & (nb - 1)], 1);
          }
          __syncthreads();
          const int per = nb / kThreads;
          int cnt = 0;
          for (int i = 0; i < per; ++i) cnt += sHist[nb - 1 - (tid * per + i)];
          int inc = cnt;  // inclusive scan of cnt over the workgroup
#pragma unroll
          for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(inc, o);
            if (lane >= o) inc += y;
          }
          if (lane == 63) sScan[wv] = inc;
          __syncthreads();
          int above = inc - cnt;
          for (int i = 0; i < wv; ++i) above += sScan[i];
          if (kk > above && kk <= above + cnt) {
            for (int i = 0; i < per; ++i) {
              const int b = nb - 1 - (tid * per + i);
              const int hb = sHist[b];
              if (kk <= above + hb) {
                sSel[0] = b;
                sSel[1] = kk - above;
                break;
              }
              above += hb;
            }
          }
          __syncthreads();
          prefix |= (uint32_t)sSel[0] << shift;
          pmask |= (uint32_t)(nb - 1) << shift;
          kk = sSel[1];
          __syncthreads();
        }
        const uint32_t tau = prefix;
        const int need = kk;  // ties at tau taken in position order
        const int seg = (n + kThreads - 1) / kThreads;
        const int j0 = min(n, tid * seg), j1 = min(n, j0 + seg);
        int gt = 0, eq = 0;
        for (int j = j0; j < j1; ++j) {
          const uint32_t x = __float_as_uint(get(j));
          gt += x > tau;
          eq += x == tau;
        }
        const int v = gt | (eq << 16);   // exclusive scan of the packed counts
        int inc = v;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(inc, o);
          if (lane >= o) inc += y;
        }
        if (lane == 63) sScan[wv] = inc;
        __syncthreads();
        int pre = inc - v;
        for (int i = 0; i < wv; ++i) pre += sScan[i];
        const int pre_gt = pre & 0xffff, pre_eq = pre >> 16;
        int out = pre_gt + min(pre_eq, need);
        int er = pre_eq;
        for (int j = j0; j < j1; ++j) {
          const uint32_t x = __float_as_uint(get(j));
          bool take = x > tau;
          if (x == tau) {
            take = er < need;
            ++er;
          }
          if (take) {
            store_coherent(idx + out, j);
            ++out;
          }
        }
      }
      const int nf = ly.forced_hi - ly.forced_lo;
      for (int t = tid; t < nf; t += kThreads) store_coherent(idx + k + t, ly.forced_lo + t);
    }
    vmem_release();
    __syncthreads();
    if (tid == 0) __hip_atomic_store(&selDone[head], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (acc) {
      // scores of the retained positions (they seed decode-phase accumulation)
      for (int m0 = tid; m0 < ly.n_keep; m0 += kThreads * 8) {
        int pos[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) pos[u] = m0 + u * kThreads < ly.n_keep ? load_coherent(idx + m0 + u * kThreads) : -1;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (pos[u] >= 0) acc[m0 + u * kThreads] = load_coherent(accsrc + pos[u]);
      }
    }
    return;
  }

  // ============================================================== stats and score items
  uint16_t* sQ = reinterpret_cast<uint16_t*>(smem);
  float* aux = reinterpret_cast<float*>(smem + kQBytes);
  const int nt_used = G * NTG;
  const int c = chunk;
  const size_t head_base = (size_t)bh * L;
  const uint16_t* khead = ly.k + head_base * kHeadDim;
  const int wave_key0 = c * kChunk + wv * kKeysPerWave;
  const bool padded_rows = (nt_used < NT) || (w != NTG * 32);

  u32x4 kf[kKDepth][8];              // ring of key tiles: the current one and kKDepth-1 ahead
#pragma unroll
  for (int d = 0; d < kKDepth - 1; ++d) load_k_frag(kf[d], khead, wave_key0 + d * 32 + ln, L, hf);
  load_q_to_lds<NT, NTG>(sQ, P, ly, s, h);
  float* sMp = aux + NG * kChunk;     // score items: per-row log-normalisers
  if (type == kItemScore) {
    // fold every chunk's (max, sum) of this head into exp2 offsets M + log2(sum) per row,
    // waiting (bounded) for chunks whose statistics are not written yet
    constexpr int kGroups = kThreads / R > 0 ? kThreads / R : 1;
    constexpr int kRowsPerPass = kThreads / kGroups;
    float* sPart = sMp + R;           // [kGroups][R][2]
    for (int r0 = 0; r0 < R; r0 += kRowsPerPass) {
      const int r = r0 + tid % kRowsPerPass;
      const int j = tid / kRowsPerPass;
      float M = NEG_INF, Ls = 0.f;
      const float* st0 = P.stats + (size_t)head * NC * R * 2 + 2 * r;
      for (int c0 = j; c0 < NC; c0 += kGroups * 8) {
        float2 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int cc = c0 + u * kGroups;
          v[u] = cc < NC ? load_coherent2(st0 + (size_t)cc * R * 2) : make_float2(NEG_INF, 0.f);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          uint32_t it = 0;
          while (unwritten(v[u].x)) {
            __builtin_amdgcn_s_sleep(2);
            v[u] = load_coherent2(st0 + (size_t)(c0 + u * kGroups) * R * 2);
            if (++it > kSpinLimit) {
              atomicOr(status, 1u);
              v[u] = make_float2(NEG_INF, 0.f);
            }
          }
          combine_ms(M, Ls, v[u].x, v[u].y);
        }
      }
      sPart[(j * R + r) * 2] = M;
      sPart[(j * R + r) * 2 + 1] = Ls;
    }
    __syncthreads();
    for (int r = tid; r < R; r += kThreads) {
      float M = sPart[r * 2], Ls = sPart[r * 2 + 1];
      for (int j = 1; j < kGroups; ++j) combine_ms(M, Ls, sPart[(j * R + r) * 2], sPart[(j * R + r) * 2 + 1]);
      // probabilities are exp2(z - M - log2 L); rows without keys (padding) get +inf -> 0
      sMp[r] = Ls > 0.f ? M + __log2f(Ls) : __builtin_inff();
    }
  }
  __syncthreads();

  if (type == kItemStats) {
    float run_m[NT], run_l[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { run_m[t] = NEG_INF; run_l[t] = 0.f; }
    // one key tile: logits for half of the row tiles at a time, then the running row
    // max / sum; lane = window row ln of tile t, registers = keys tile_key0 + 8(r/4) + 4hf + r%4
    auto tile = [&](const u32x4 (&kft)[8], int tile_key0) {
      const bool need_mask = padded_rows || (tile_key0 + 32 > L - w);
#pragma unroll
      for (int half = 0; half < NT / kRowTilesPerPass; ++half) {
        constexpr int NH = kRowTilesPerPass;
        f32x16 acc[NH];
        mfma_tile<NH, false>(acc, kft, sQ, ln, hf, half * NH, nt_used);
#pragma unroll
        for (int i = 0; i < NH; ++i) {
          const int t = half * NH + i;
          if (t >= nt_used) continue;
          if (need_mask) mask_rows_lane<NTG>(acc[i], t, ln, hf, tile_key0, G, w, L);
          float tm = acc[i][0];
#pragma unroll
          for (int r = 1; r < 16; ++r) tm = fmaxf(tm, acc[i][r]);
          if (tm == NEG_INF) continue;
          const float nm = fmaxf(run_m[t], tm * sl2);
          float sm = run_l[t] * __builtin_amdgcn_exp2f(run_m[t] - nm);
#pragma unroll
          for (int r = 0; r < 16; ++r) sm += __builtin_amdgcn_exp2f(fmaf(acc[i][r], sl2, -nm));
          run_m[t] = nm;
          run_l[t] = sm;
        }
      }
    };
#pragma unroll 1
    for (int base = 0; base < kTilesPerWave; base += kKDepth) {
#pragma unroll
      for (int i = 0; i < kKDepth; ++i) {
        const int kt = base + i;
        // keys kKDepth-1 tiles ahead load while this tile is multiplied and exponentiated
        if (kt + kKDepth - 1 < kTilesPerWave)
          load_k_frag(kf[(i + kKDepth - 1) % kKDepth], khead, wave_key0 + (kt + kKDepth - 1) * 32 + ln, L, hf);
        if (wave_key0 + kt * 32 < L) tile(kf[i], wave_key0 + kt * 32);
      }
    }
    // fold the two lanes that share a row, then the four waves
    float* sRed = aux;  // [kWaves][R][2]
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float m2 = __shfl_xor(run_m[t], 32), l2 = __shfl_xor(run_l[t], 32);
      float M = run_m[t], Ls = run_l[t];
      combine_ms(M, Ls, m2, l2);
      if (hf == 0) {
        sRed[(wv * R + t * 32 + ln) * 2] = M;
        sRed[(wv * R + t * 32 + ln) * 2 + 1] = Ls;
      }
    }
    __syncthreads();
    float* stat = P.stats + ((size_t)head * NC + c) * R * 2;
    for (int r = tid; r < R; r += kThreads) {
      float M = NEG_INF, Ls = 0.f;
#pragma unroll
      for (int v = 0; v < kWaves; ++v) combine_ms(M, Ls, sRed[(v * R + r) * 2], sRed[(v * R + r) * 2 + 1]);
      store_coherent2(stat + 2 * r, M, Ls);
    }
    return;
  }

  // ---------------------------------------------------------------- score item
  float* sA = aux;  // [NG][kChunk] window column sums of this chunk per query head
  // one key tile: probabilities for half of the row tiles at a time and their column sums per
  // query head; lane = key tile_key0 + ln, registers = rows t*32 + 8(r/4) + 4hf + r%4
  auto tile = [&](const u32x4 (&kft)[8], int tile_key0, int local0) {
    const int key = tile_key0 + ln;
    const bool need_mask = padded_rows || (tile_key0 + 32 > L - w);
    float col[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) col[g] = 0.f;
#pragma unroll
    for (int half = 0; half < NT / kRowTilesPerPass; ++half) {
      constexpr int NH = kRowTilesPerPass;
      f32x16 acc[NH];
      mfma_tile<NH, true>(acc, kft, sQ, ln, hf, half * NH, nt_used);
#pragma unroll
      for (int i = 0; i < NH; ++i) {
        const int t = half * NH + i;
        if (t >= nt_used) continue;
        float mp[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 v = *reinterpret_cast<const float4*>(sMp + t * 32 + 8 * q + 4 * hf);
          mp[4 * q] = v.x; mp[4 * q + 1] = v.y; mp[4 * q + 2] = v.z; mp[4 * q + 3] = v.w;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = __builtin_amdgcn_exp2f(fmaf(acc[i][r], sl2, -mp[r]));
        if (need_mask) mask_rows_regs<NTG>(acc[i], t, hf, key, G, w, L);
        float cs = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) cs += acc[i][r];
        col[t / NTG] += cs;
      }
    }
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const float v = col[g] + __shfl_xor(col[g], 32);
      if (hf == 0 && g < G) sA[g * kChunk + local0 + ln] = v;
    }
  };
#pragma unroll 1
  for (int base = 0; base < kTilesPerWave; base += kKDepth) {
#pragma unroll
    for (int i = 0; i < kKDepth; ++i) {
      const int kt = base + i;
      if (kt + kKDepth - 1 < kTilesPerWave)
        load_k_frag(kf[(i + kKDepth - 1) % kKDepth], khead, wave_key0 + (kt + kKDepth - 1) * 32 + ln, L, hf);
      if (wave_key0 + kt * 32 < L) tile(kf[i], wave_key0 + kt * 32, wv * kKeysPerWave + kt * 32);
    }
  }
  __syncthreads();

  // group mean (unpooled), in-chunk max-pool (SnapKV), scores and chunk-edge values
  const int cbase = c * kChunk;
  float* Srow = P.S + (size_t)head * L;
  for (int kl = tid; kl < kChunk; kl += kThreads) {
    const int key = cbase + kl;
    if (key >= L) break;
    float su = 0.f;
    for (int g = 0; g < G; ++g) su += sA[g * kChunk + kl];
    su = su / (float)G;
    if (snap) {
      const int npre = L - w;
      float sc = su;
      if (key < npre) {
        const int ph = P.pool_half;
        const int lo = max(key - ph, cbase), hi = min(min(key + ph, cbase + kChunk - 1), npre - 1);
        sc = 0.f;
        for (int g = 0; g < G; ++g) {
          float m = NEG_INF;
          for (int t = lo; t <= hi; ++t) m = fmaxf(m, sA[g * kChunk + t - cbase]);
          sc += m;
        }
        sc = sc / (float)G;
      }
      store_coherent(Srow + key, sc);
      if (P.want_unpooled) store_coherent(P.Su + (size_t)head * L + key, su);
    } else {
      store_coherent(Srow + key, su);
    }
  }
  if (snap && P.pool_half > 0) {
    const int E = 4 * P.pool_half, twoP = 2 * P.pool_half;
    float* ed = P.edge + ((size_t)head * NC + c) * G * E;
    for (int e = tid; e < G * E; e += kThreads) {
      const int g = e / E, o = e - g * E;
      const int kl = o < twoP ? o : kChunk - twoP + (o - twoP);
      store_coherent(ed + e, (cbase + kl < L) ? sA[g * kChunk + kl] : 0.f);
    }
  }
}

template <int NT, int NTG>
int resident_groups() {
  static int cached = -1;
  if (cached < 0) {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, evict_kernel<NT, NTG>, kThreads, 0) != hipSuccess ||
        per_cu < 1)
      per_cu = 1;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
      cus = 256;
    cached = per_cu * cus;
  }
  return cached;
}

template <int NT, int NTG>
int launch_evict(PrefillLaunch P, hipStream_t st, void* stream) {
  const int nH = P.batch * P.n_scored * P.n_kv_heads;
  // Lags between a head's phases, in steps: about one resident round of workgroups between its
  // stats and score items and between its score and select items (so those items rarely wait,
  // and the score items still find the head's K in the on-die caches); the gather items only
  // wait for the one select item.
  const int per_step = 2 * P.n_chunks + 1 + kGatherParts;
  const int round = (resident_groups<NT, NTG>() + per_step - 1) / per_step;
  P.lag_score = round + 1;
  P.lag_select = round + 1;
  P.lag_gather = round / 3 + 1;
  const int64_t scored = nH > 0 ? (int64_t)nH * (2 * P.n_chunks + 1 + kGatherParts) : 0;
  const int64_t copies = (int64_t)P.n_unscored * P.batch * P.n_kv_heads * kGatherParts;
  const int64_t total = scored + copies;
  if (total <= 0) return 0;
  if (total > 0x7fffffff) return (int)hipErrorInvalidValue;
  P.n_tickets = (int)total;
  profile_mark(kStageScore, false, stream);
  evict_kernel<NT, NTG><<<(unsigned)total, kThreads, 0, st>>>(P);
  profile_mark(kStageScore, true, stream);
  return 0;
}

}  // namespace

int launch_prefill(const PrefillLaunch& P, int row_tiles, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int nH = P.batch * P.n_scored * P.n_kv_heads;
  {
    const int nc = 2 + nH;
    const int64_t n_fill = nH > 0 ? P.fill_vec4 : 0;
    int64_t blocks = (std::max<int64_t>(nc, n_fill) + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    profile_mark(kStageZero, false, stream);
    reset_workspace<<<(unsigned)blocks, 256, 0, st>>>(P.counters, nc, reinterpret_cast<u32x4*>(P.stats), n_fill);
    profile_mark(kStageZero, true, stream);
  }
  int err = 0;
  const int ntg = P.row_tiles_per_group;
  if (row_tiles == 4 && ntg == 1) err = launch_evict<4, 1>(P, st, stream);
  else if (row_tiles == 4 && ntg == 2) err = launch_evict<4, 2>(P, st, stream);
  else if (row_tiles == 4) err = launch_evict<4, 4>(P, st, stream);
  else if (ntg == 1) err = launch_evict<8, 1>(P, st, stream);
  else if (ntg == 2) err = launch_evict<8, 2>(P, st, stream);
  else if (ntg == 4) err = launch_evict<8, 4>(P, st, stream);
  else err = launch_evict<8, 8>(P, st, stream);
  if (err) return err;
  return (int)hipGetLastError();
}

}  // namespace rkv
