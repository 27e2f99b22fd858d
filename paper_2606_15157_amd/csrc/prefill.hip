// Prefill prompt compression for gfx950 (CDNA4).
//
// Per (sequence, scored layer, KV head) -- a "job" -- the window scores are (Section 2.1, the
// SnapKV and H2O retention rules the route composes)
//   A[g][j] = sum_i softmax_j(Q[g,i] . K[j] / sqrt(d))      (w window rows per query head g)
//   S[j]    = mean_g maxpool(A[g])[j]  (SnapKV)  or  mean_g A[g][j]  (H2O)
// A row's softmax is normalised over every key while the window sum runs over rows, so a row's
// normaliser is known only once every key of the job has been seen.  Work items are (job,
// slice of 128 keys).
//   prepare + pipelined scoring kernel (four row tiles, at most 64 slices per job): persistent,
//     one eight-wave workgroup per CU, four items in flight; each slice streams its K tile
//     once, publishes per-row sums against a fixed per-row reference logit, and turns its
//     exponentials into probabilities once the job's sums are in (two levels: per slice group,
//     then per job; the kernel's own comment below has the schedule);
//   window kernels (window.hip; longer prompts and eight row tiles): row normalisers, then
//     column sums, each streaming K once;
//   select kernels (one workgroup per job): repair the pooled score next to slice borders (or
//     rescore a job flagged for a reference overflow exactly), find the k-th largest score with
//     at most three radix-histogram passes and write the retained positions in ascending order;
//   gather kernel: copies the retained K and V rows.
//
// Data handed between workgroups of one launch goes through device-coherent loads and stores
// (they bypass the XCD-local caches) over a NaN "not stored" mark, so no agent-scope fence
// (which would flush and invalidate L2) is needed.  Every wait is bounded: on time-out the
// workspace status word is set and the kernel carries on.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <math.h>

#include <algorithm>

#include "lds_dma.h"
#include "rkv_internal.h"

namespace rkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;            // 4 waves, one per SIMD
constexpr int kWaves = kThreads / 64;
static_assert(kSlice == kWaves * 32, "one 32-key tile per wave");
constexpr uint32_t kSpinLimit = 1u << 21;
constexpr int kHistBins = 2048;
constexpr int kSelectLds = 128 * 1024;   // dynamic LDS of the select kernel (scores cached up to ~30K keys)

__device__ __forceinline__ void store_coherent2(float* p, float a, float b) {
  const uint64_t v = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Index of this wave in the workgroup, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

// Waits for every outstanding load of this wave.  Used right after a batch of loads whose values
// feed predicated stores: with loads still pending at the branch joins, the compiler would wait
// for all memory operations (earlier stores included) before every one of those stores.
__device__ __forceinline__ void loads_done() { __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8)); }

// Zeroes the counters (the status word at counters[0] only in the call's first launch group, so
// that it covers the whole call) before the window scoring kernels.
__global__ void reset_counters(uint32_t* counters, int n, int clear_status) {
  const int i0 = blockIdx.x * blockDim.x + threadIdx.x, stride = gridDim.x * blockDim.x;
  for (int i = i0; i < n; i += stride)
    if (i > 0 || clear_status) counters[i] = 0u;
}

// ---------------------------------------------------------------------------------------------
// Cross-lane sums over the 32 window rows held by the lanes of each half-wave.
// ---------------------------------------------------------------------------------------------
// Sum of an integer over the 16 lanes of each DPP row (every lane of the row gets it).
__device__ __forceinline__ int row16_sum(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x128, 0xf, 0xf, false);   // row_ror:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x124, 0xf, 0xf, false);   // row_ror:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x122, 0xf, 0xf, false);   // row_ror:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x121, 0xf, 0xf, false);   // row_ror:1
  return x;
}
// Minimum / maximum of an unsigned value over the 16 lanes of each DPP row (every lane gets it).
__device__ __forceinline__ uint32_t row16_umin(uint32_t x) {
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x128, 0xf, 0xf, false));   // row_ror:8
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x124, 0xf, 0xf, false));   // row_ror:4
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x122, 0xf, 0xf, false));   // row_ror:2
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x121, 0xf, 0xf, false));   // row_ror:1
  return x;
}
__device__ __forceinline__ uint32_t row16_umax(uint32_t x) {
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x128, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x124, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x122, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x121, 0xf, 0xf, false));
  return x;
}
// Inclusive prefix sum over the 64 lanes of a wave: shifts by 1, 2, 4, 8 inside each 16-lane row
// (lanes shifted in from outside the row read 0), then each row's total carried into the rows
// after it (row_bcast:15 into rows 1 and 3, row_bcast:31 into rows 2 and 3).
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);    // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);    // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);    // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);    // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);   // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);   // row_bcast:31
  return x;
}
template <int CTRL>
__device__ __forceinline__ float dppf(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}
// One halving step between lane pairs (permutation CTRL pairs each lane with one whose `bit` is
// the opposite): value pair (a, b) becomes a-sum in lanes with bit 0 and b-sum in lanes with bit 1.
template <int CTRL, int N, int V>
__device__ __forceinline__ void dpp_halve(float (&v)[V], int bit) {
  if constexpr (N == 1) {
    v[0] += dppf<CTRL>(v[0]);
  } else {
#pragma unroll
    for (int i = 0; i < N / 2; ++i) {
      const float a = v[2 * i], b = v[2 * i + 1];
      const float keep = bit ? b : a, send = bit ? a : b;
      v[i] = keep + dppf<CTRL>(send);
    }
  }
}
// Work item of the pipelined kernel: the item index it = first + t n_wg names job it / nsl and
// position s0 = it % nsl, and the item processes slice (s0 + job) % nsl.  The rotation moves a
// job's last slice (the one holding the observation window, slower because of its masks) to a
// different workgroup for every job, so no workgroup is every job's straggler.
struct PipeRef {
  int job, slice, s0, jm, slot, s, h;   // jm = job % nsl
};
__device__ __forceinline__ PipeRef pipe_item(int64_t it, int nsl, int B, int Hkv) {
  PipeRef r;
  r.job = (int)(it / nsl);
  r.s0 = (int)(it - (int64_t)r.job * nsl);
  r.jm = r.job % nsl;
  r.slice = r.s0 + r.jm >= nsl ? r.s0 + r.jm - nsl : r.s0 + r.jm;
  r.h = r.job % Hkv;
  r.s = (r.job / Hkv) % B;
  r.slot = r.job / (Hkv * B);
  return r;
}
// Moves an item forward by n_wg items (dj jobs and ds positions) without divisions.
__device__ __forceinline__ void pipe_advance(PipeRef& r, int dj, int ds, int nsl, int B, int Hkv) {
  r.s0 += ds;
  int j = dj;
  if (r.s0 >= nsl) {
    r.s0 -= nsl;
    ++j;
  }
  r.job += j;
  r.jm += j;
  while (r.jm >= nsl) r.jm -= nsl;
  r.slice = r.s0 + r.jm >= nsl ? r.s0 + r.jm - nsl : r.s0 + r.jm;
  r.h += j;
  while (r.h >= Hkv) {
    r.h -= Hkv;
    if (++r.s == B) {
      r.s = 0;
      ++r.slot;
    }
  }
}

// Workgroup barrier for data handed over through LDS only: this wave's LDS operations retire
// (lgkmcnt 0), then s_barrier.  Unlike __syncthreads it does not wait for the wave's vector
// memory operations (the workgroup-scope release fence does), so prefetches, stores and polls
// stay in flight across it.  LDS written by LDS DMA is covered by the issuing wave's own vmcnt
// wait before it reaches the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xc07f);   // vmcnt 63 (no wait), expcnt 7 (no wait), lgkmcnt 0
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// ---------------------------------------------------------------------------------------------
// Pipelined scoring against a per-row reference (four row tiles, one eight-wave workgroup per
// CU, four items in flight).
//
// Reference.  The softmax of a window row is shift-invariant, so the exponentials may be taken
// against any per-row constant c_i that keeps them in range.  c_i is the larger of the row's
// logit with its own key (position L - w + i, always visible) and with the first key; both are
// true logits of the row, so e_ij = exp2((z_ij - c_i) log2(e) / sqrt(d)) <= 2^127 unless some
// key beats the reference by more than 88 (natural log units), and the row sum Z_i >= 1 (the
// reference key contributes 1).  Then p_ij = e_ij / Z_i: a slice publishes plain row sums, the
// normaliser is their sum, and no running maximum is needed.  A non-finite Z_i is reported in
// the status word (bit 1).
//
// Layout.  16x16x32 bf16 MFMA with the queries as the A operand: in every 16 x 16 tile lane l
// holds key l % 16 and rows 4 (l / 16) + 0..3.  Wave wv takes keys 32 (wv % 4) + [0, 32) of the
// item's 128-key slice (two key sub-tiles) and rows 64 (wv / 4) + [0, 64) (four row sub-tiles):
// 8 tiles, 32 exponentials per lane.  Sums over window rows are then register-local plus two
// permlane swaps; sums over keys (row statistics) take four DPP steps inside each row of 16
// lanes.
//
// Normalisers, in two levels.  Each slice stores its 128 row sums (level 0).  A job's slices form
// up to kPipeGroups groups of gs consecutive slices; the workgroup that scores a group's first
// slice sums the group's row sums into a partial (level 1), and every workgroup that scores a
// slice of the job sums the job's partials (level 2).  Every hop is store -> load with "not
// stored" marked NaN, no counters; the additions run in a fixed order, so results are
// reproducible.  Per item a workgroup reads 4 KiB of partials (and a group's first workgroup
// 4 KiB of row sums) instead of the job's 32 KiB of row sums.
//
// Schedule of iteration t (item t enters phase A, item t - 3 phase B, each in its own register
// set; no wait is for an operation issued in the same iteration).  There is no barrier between
// one iteration's score stores and the next phase A: every buffer phase A and MID touch was
// handed on by B1.5 or B2 of the previous iteration, and the score stores read the sColP buffer
// of their own iteration's parity, so a wave whose SIMD partner is still issuing DMA starts the
// next item's MFMAs at once:
//   A     logits (fragments read two MFMA pairs ahead), exponentials, per-row partial sums per
//         key tile into sStat
//   MID   every wave: all its earlier memory operations have completed; waves 0-3: the partials
//         of item t - 3's job (loaded at the end of iteration t - 1; re-read while any is still
//         NaN) -> reciprocal normalisers in sAlpha; the loads of item t - 1's group's row sums
//         where this workgroup sums that group
//   B1.5
//   wave 0: store item t's row sums
//   B     item t - 3: probabilities, sums over the window rows per query head (or group) into
//         sColP[t % 2]
//   B2
//   waves 0-3: the partial of item t - 1's group (where this workgroup sums it: its row sums
//         re-read while any is NaN), the scores of item t - 3, the loads of item t - 2's
//         partials; waves 4-7: LDS DMA of item t + 2 into the buffer item t has just left
// The margins: row sums stored at B1.5 of iteration u are loaded at MID of u + 1; partials
// stored at the end of u + 1 are loaded at the end of u + 2, about an iteration later each.
// Progress: every wait is for a store that its workgroup makes earlier in its own sequence than
// the waiting point (a job's slices sit in at most two consecutive iterations because a job has
// no more slices than there are workgroups), so with every workgroup resident no wait is on a
// later one.
// ---------------------------------------------------------------------------------------------
constexpr int kPipeWaves = 8;
constexpr int kPipeThreads = kPipeWaves * 64;
constexpr int kPipeShortItems = 4;   // items per workgroup up to which the short form runs

typedef float f32x4v __attribute__((ext_vector_type(4)));


// Minus the reference logit of every row of every scored job, and the per-pass resets: the
// status word, the job's slices' row sums and its partials ("not stored": NaN).
// Sixteen workgroups of 128 threads per job, each with eight of the rows and a sixteenth of the
// resets (many small workgroups: the kernel is a few dependent memory round trips).
constexpr int kPrepParts = 16, kPrepThreads = 128;
template <int NTH>
__global__ __launch_bounds__(kPrepThreads) void prepare_kernel(const PrefillLaunch P) {
  constexpr int R = 128;
  // workgroup q of the job takes rows 8 q + [0, 8) and a sixteenth of the fill
  constexpr int kParts = kPrepParts;
  const int tid = threadIdx.x, job = blockIdx.x / kParts, q = blockIdx.x % kParts;
  const int Hkv = P.n_kv_heads, B = P.batch, L = P.seq_len, w = P.window, G = P.group, Hq = P.n_q_heads;
  const int h = job % Hkv, s = (job / Hkv) % B, slot = job / (Hkv * B);
  const PrefillLayer& ly = P.layer[P.slot_layer[slot]];
  if (blockIdx.x == 0 && tid == 0 && P.first_group) P.counters[0] = 0u;   // once per call
  if (q == 0 && tid == 0) P.counters[(size_t)kCounterStride * (1 + job) + 1] = 0u;   // the job's repair flag
  // 16 lanes per row, lane c taking 16-byte chunk c of the query, the row's own key and key 0
  // (each load instruction reads whole 256-byte rows); the loads are issued before the fill's
  // stores so that their latency overlaps them
  const int c = tid & 15;
  const u32x4* ks = reinterpret_cast<const u32x4*>(ly.k + (size_t)(s * Hkv + h) * L * kHeadDim) + c;
  const int r = 8 * q + (tid >> 4);
  const int g = r / (NTH * 32), ii = r - g * (NTH * 32);
  const bool valid = g < G && ii < w;
  u32x4 qa = {0u, 0u, 0u, 0u}, da = qa, sa = qa;
  if (valid) {
    qa = reinterpret_cast<const u32x4*>(ly.q + ((size_t)(s * Hq + h * G + g) * w + ii) * kHeadDim)[c];
    da = ks[(size_t)(L - w + ii) * 16];
    sa = ks[0];
  }
  {
    // every slice's row sums "not stored yet" (NaN): the consumers check them
    u32x4* st = reinterpret_cast<u32x4*>(P.stats + (size_t)job * P.n_slices * R);
    const u32x4 nan4 = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};
    for (int i = tid + kPrepThreads * q; i < P.n_slices * R / 4; i += kPrepThreads * kParts) st[i] = nan4;
    // and the job's level-1 partials
    u32x4* pt = reinterpret_cast<u32x4*>(P.part + (size_t)job * kPipeGroups * R);
    for (int i = tid + kPrepThreads * q; i < kPipeGroups * R / 4; i += kPrepThreads * kParts) pt[i] = nan4;
  }
  float zd = 0.f, zs = 0.f;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const float q0 = __uint_as_float(qa[u] << 16), q1 = __uint_as_float(qa[u] & 0xffff0000u);
    zd = fmaf(q0, __uint_as_float(da[u] << 16), zd);
    zd = fmaf(q1, __uint_as_float(da[u] & 0xffff0000u), zd);
    zs = fmaf(q0, __uint_as_float(sa[u] << 16), zs);
    zs = fmaf(q1, __uint_as_float(sa[u] & 0xffff0000u), zs);
  }
  // sums over the 16 lanes of the row: rotations by 8, 4, 2, 1 inside each 16-lane DPP row
  zd += dppf<0x128>(zd);
  zs += dppf<0x128>(zs);
  zd += dppf<0x124>(zd);
  zs += dppf<0x124>(zs);
  zd += dppf<0x122>(zd);
  zs += dppf<0x122>(zs);
  zd += dppf<0x121>(zd);
  zs += dppf<0x121>(zs);
  if (c == 0) P.ncl[(size_t)job * R + r] = valid ? -fmaxf(zd, zs) : 0.f;
}

// Reduce-scatter of 16 values over the 16 lanes of each row: afterwards lane l holds the sum of
// value 8 b0 + 4 b1 + 2 b2 + b3 (b_k = bit k of l) over its row.
__device__ __forceinline__ void reduce_scatter16(float (&v)[16], int lane) {
  dpp_halve<0x128, 16, 16>(v, (lane >> 3) & 1);   // row_ror:8        -> lane l ^ 8
  dpp_halve<0x141, 8, 16>(v, (lane >> 2) & 1);    // row_half_mirror  -> 7 - l within 8
  dpp_halve<0x4E, 4, 16>(v, (lane >> 1) & 1);     // quad_perm [2,3,0,1] -> l ^ 2
  dpp_halve<0xB1, 2, 16>(v, lane & 1);            // quad_perm [1,0,3,2] -> l ^ 1
}
__device__ __forceinline__ int rs16_sel(int lane) {
  return ((lane & 1) << 3) | (((lane >> 1) & 1) << 2) | (((lane >> 2) & 1) << 1) | ((lane >> 3) & 1);
}
__device__ __forceinline__ bf16x8 frag16(const uint16_t* base, int row, int chunk) {
  return *reinterpret_cast<const bf16x8*>(base + (row * 16 + (chunk ^ (row & 15))) * 8);
}

// SHORT: every workgroup has at most a few items (short prompts, few layers); then the phases of
// the pipeline's fill and drain iterations, which only run on stale data, are skipped (in long
// runs they stay unconditional: the loop's code is then the tighter one).
template <int NTH, bool SHORT>
__global__ __launch_bounds__(kPipeThreads, 1) void score_pipe_kernel(const PrefillLaunch P, int n_wg) {
  constexpr int R = 128;
  __shared__ __attribute__((aligned(16))) uint16_t sQ[2][R * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kSlice * kHeadDim];
  __shared__ __attribute__((aligned(16))) float sNcl[2][R];
  __shared__ __attribute__((aligned(16))) float sAlpha[R];
  __shared__ float sStat[4][R];
  __shared__ float sColPb[2][2][2][kSlice];   // two buffers, by iteration parity
  float (*sColP)[2][kSlice] = sColPb[0];

  const int tid = threadIdx.x, lane = tid & 63, wv = wave_id(), lg = lane >> 4, l16 = lane & 15;
  const int kt = wv & 3, rh = wv >> 2;
  const int L = P.seq_len, w = P.window, G = P.group, Hkv = P.n_kv_heads, B = P.batch, Hq = P.n_q_heads;
  const int nsl = P.n_slices;
  const int n_jobs = B * P.n_window * Hkv;
  const int64_t n_items = (int64_t)n_jobs * nsl;
  const float sl2 = P.scale_log2;
  const float inv_g = 1.f / (float)G;
  uint32_t* status = P.counters;
  const bool padded_rows = (G * NTH < 4) || (w != NTH * 32);

  const int64_t first = blockIdx.x;
  if (first >= n_items) return;
  const int T = (int)((n_items - 1 - first) / n_wg + 1);
  const int dj = n_wg / nsl, ds = n_wg - dj * nsl;   // item stride n_wg in (jobs, slices)
  bool gave_up = false;   // a wait of this wave timed out (status set): no further waits

  // ---- waves 4-7: the item's query block, K tile and reference logits into buffer b.
  // Instruction u (0..15) of wave 4 + dw moves 1 KiB: rows (u < 8) or keys (u >= 8)
  // 16 (u % 8) + 4 dw + [0, 4); lane l fills row / key 16 (u % 8) + lrow, chunk position l % 16,
  // with lrow = 4 dw + l / 16 and source chunk (l % 16) ^ lrow (the swizzle of issue_q_to_lds).
  // The lane's byte offset is the same for every instruction; wave 4 also moves the references.
  const int lrow = 4 * (wv & 3) + (lane >> 4);
  const uint32_t lane_off = (uint32_t)lrow * 256u + (uint32_t)((lane & 15) ^ lrow) * 16u;
  auto issue_dma = [&](const PipeRef& j, int b) {
    const PrefillLayer& ly = P.layer[j.slot];
    const char* qjob = reinterpret_cast<const char*>(ly.q + (size_t)(j.s * Hq + j.h * G) * w * kHeadDim);
    const char* khead = reinterpret_cast<const char*>(ly.k + (size_t)(j.s * Hkv + j.h) * L * kHeadDim);
    const int key0 = j.slice * kSlice;
    const uint32_t q_lds = lds_addr(&sQ[b][4 * (wv & 3) * kHeadDim]);
    const uint32_t k_lds = lds_addr(&sK[b][4 * (wv & 3) * kHeadDim]);
    // common case: a uniform base per instruction (scalar arithmetic) and the lane's fixed offset
    if (__builtin_expect(!padded_rows, 1)) {
      // w = 32 NTH rows per head and G NTH = 4: instruction u reads rows 16 u + lrow, 4 KiB apart
#pragma unroll
      for (int u = 0; u < 8; u += 2) dma16s_pair(qjob + 4096u * u, lane_off, q_lds + 4096u * u);
    } else {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int g = u / (2 * NTH), ii0 = 16 * (u % (2 * NTH));
        const bool ok = g < G && ii0 + lrow < w;
        const uint32_t off = ok ? (uint32_t)(g * w + ii0) * 256u + lane_off
                                : (uint32_t)((lane & 15) ^ lrow) * 16u;   // padding rows repeat row 0
        dma16(qjob + off, q_lds + 16u * kHeadDim * 2u * u);
      }
    }
    const bool tail = key0 + kSlice > L;
    if (__builtin_expect(!tail, 1)) {
      const char* kslice = khead + (size_t)key0 * 256u;
#pragma unroll
      for (int u = 0; u < 8; u += 2) dma16s_pair(kslice + 4096u * u, lane_off, k_lds + 4096u * u);
    } else {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int key = min(key0 + 16 * u + lrow, L - 1);
        dma16(khead + (size_t)key * 256u + (uint32_t)((lane & 15) ^ lrow) * 16u, k_lds + 16u * kHeadDim * 2u * u);
      }
    }
    if (wv == 4) {
      // the job's 128 reference logits: lanes 0-31 move 16 bytes each (the DMA writes only the
      // active lanes' 16-byte pieces)
      const uint32_t n_lds = lds_addr(&sNcl[b][0]);
      if (lane < 32) dma16(P.ncl + (size_t)j.job * R + 4 * lane, n_lds);
    }
  };
  // ---- phase A: e = exp2((z - c) log2(e)/sqrt(d)) for tile (rs, ks): row rh*64 + 16 rs + 4 lg + i,
  // key key0 + 32 kt + 16 ks + l16; per-row partial sums over this wave's 32 keys into sStat[kt]
  auto phase_a = [&](const PipeRef& j, int b, f32x4v (&e)[4][2]) {
    const uint16_t* q = sQ[b];
    const uint16_t* k = sK[b];
#pragma unroll
    for (int rs = 0; rs < 4; ++rs) {
      const f32x4v c4 = *reinterpret_cast<const f32x4v*>(&sNcl[b][rh * 64 + rs * 16 + 4 * lg]);
      e[rs][0] = c4;
      e[rs][1] = c4;
    }
    // software pipeline over the 16 (k-step, row tile) MFMA pairs: the query fragment of pair p
    // is read two pairs ahead, the two key fragments of k-step st + 1 at the first pair of st.
    // The fragment addresses come from an opaque copy of the thread index, so that they are
    // recomputed per item instead of being held in registers across the loop.
    int tv = threadIdx.x;
    asm volatile("" : "+v"(tv));
    const int l16v = tv & 15, lgv = (tv >> 4) & 3;
    const char* qrow = reinterpret_cast<const char*>(q) + (rh * 64 + l16v) * 256;
    const char* krow = reinterpret_cast<const char*>(k) + (kt * 32 + l16v) * 256;
    // 16-byte chunk 4 st + lg of a row sits at chunk position (4 st + lg) ^ (row % 16)
    auto xo = [&](int st) { return ((4 * st + lgv) ^ l16v) << 4; };
    auto qfrag = [&](int pp) { return *reinterpret_cast<const bf16x8*>(qrow + (pp & 3) * 4096 + xo(pp >> 2)); };
    auto kfrag = [&](int st, int ks) { return *reinterpret_cast<const bf16x8*>(krow + ks * 4096 + xo(st)); };
    bf16x8 kf[2][2], qf[3];
    kf[0][0] = kfrag(0, 0);
    kf[0][1] = kfrag(0, 1);
    qf[0] = qfrag(0);
    qf[1] = qfrag(1);
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);   // DS reads: the references, k-step 0
#pragma unroll
    for (int pp = 0; pp < 16; ++pp) {
      const int st = pp >> 2, rs = pp & 3;
      const bool rq = pp + 2 < 16, rk = rs == 0 && st < 3;
      if (rq) qf[(pp + 2) % 3] = qfrag(pp + 2);
      if (rk) {
        kf[(st + 1) & 1][0] = kfrag(st + 1, 0);
        kf[(st + 1) & 1][1] = kfrag(st + 1, 1);
      }
      if (rq && rk) __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
      else if (rk) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      else if (rq) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      e[rs][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[pp % 3], kf[st & 1][0], e[rs][0], 0, 0, 0);
      e[rs][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[pp % 3], kf[st & 1][1], e[rs][1], 0, 0, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);   // MFMA
    }
    __builtin_amdgcn_sched_barrier(0);
    const int key_w0 = j.slice * kSlice + kt * 32;
    if (__builtin_expect(padded_rows || key_w0 + 31 > L - w, 0)) {
      // rare tiles (reaching into the window or past the prompt, or padding rows): logits of
      // keys a row does not see become -inf.  Lane quantities come from an opaque copy of the
      // thread index so that the compiler keeps none of this live across the loop.
      int tv = tid;
      asm volatile("" : "+v"(tv));
      const int lgv = (tv & 63) >> 4, kv = key_w0 + (tv & 15);
#pragma unroll
      for (int rs = 0; rs < 4; ++rs)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = rh * 64 + rs * 16 + 4 * lgv + i;
          const int g = row / (NTH * 32), ii = row - g * (NTH * 32);
          const int last = (g < G && ii < w) ? min(L - 1, L - w + ii) : -1;
          if (kv > last) e[rs][0][i] = -__builtin_inff();
          if (kv + 16 > last) e[rs][1][i] = -__builtin_inff();
        }
    }
    float v[16];
#pragma unroll
    for (int rs = 0; rs < 4; ++rs)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x0 = __builtin_amdgcn_exp2f(e[rs][0][i] * sl2);
        const float x1 = __builtin_amdgcn_exp2f(e[rs][1][i] * sl2);
        e[rs][0][i] = x0;
        e[rs][1][i] = x1;
        v[4 * rs + i] = x0 + x1;
      }
    reduce_scatter16(v, lane);
    const int sel = rs16_sel(l16);
    sStat[kt][rh * 64 + (sel >> 2) * 16 + 4 * lg + (sel & 3)] = v[0];
  };

  // ---- phase B: p = e / Z; sums over the window rows into sColP[rh][slot][key]: slot = query
  // head within the row half (SnapKV, one row tile per head), else 0 (one head per row half, or
  // the partial group / head sum of this row half)
  auto phase_b = [&](const PipeRef& j, f32x4v (&e)[4][2]) {
    // the slot is clamped: phase B also runs, with its results unused, for items past the end
    const bool snap = P.layer[min(j.slot, P.n_window - 1)].rule == RKV_SNAPKV;
    f32x4v a4[4];
#pragma unroll
    for (int rs = 0; rs < 4; ++rs) a4[rs] = *reinterpret_cast<const f32x4v*>(&sAlpha[rh * 64 + rs * 16 + 4 * lg]);
    if (snap && NTH == 1) {
      float c[4] = {0.f, 0.f, 0.f, 0.f};   // (slot, ks) = (0,0) (0,1) (1,0) (1,1)
#pragma unroll
      for (int rs = 0; rs < 4; ++rs)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          c[2 * (rs >> 1)] = fmaf(a4[rs][i], e[rs][0][i], c[2 * (rs >> 1)]);
          c[2 * (rs >> 1) + 1] = fmaf(a4[rs][i], e[rs][1][i], c[2 * (rs >> 1) + 1]);
        }
      const auto p0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(c[0]), __float_as_uint(c[1]), false, false);
      const auto p1 = __builtin_amdgcn_permlane32_swap(__float_as_uint(c[2]), __float_as_uint(c[3]), false, false);
      const float w0 = __uint_as_float(p0[0]) + __uint_as_float(p0[1]);
      const float w1 = __uint_as_float(p1[0]) + __uint_as_float(p1[1]);
      const auto p2 = __builtin_amdgcn_permlane16_swap(__float_as_uint(w0), __float_as_uint(w1), false, false);
      const float x = __uint_as_float(p2[0]) + __uint_as_float(p2[1]);
      // lane group lg holds (slot, ks) = (lg & 1, lg >> 1)
      sColP[rh][lg & 1][kt * 32 + (lg >> 1) * 16 + l16] = x;
    } else {
      float c[2] = {0.f, 0.f};
#pragma unroll
      for (int rs = 0; rs < 4; ++rs)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          c[0] = fmaf(a4[rs][i], e[rs][0][i], c[0]);
          c[1] = fmaf(a4[rs][i], e[rs][1][i], c[1]);
        }
      const auto p0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(c[0]), __float_as_uint(c[1]), false, false);
      const float w0 = __uint_as_float(p0[0]) + __uint_as_float(p0[1]);
      const auto p1 = __builtin_amdgcn_permlane16_swap(__float_as_uint(w0), __float_as_uint(w0), false, false);
      const float x = __uint_as_float(p1[0]) + __uint_as_float(p1[1]);
      // lane groups 0, 1 hold ks = 0, groups 2, 3 hold ks = 1 (each twice)
      if ((lg & 1) == 0) sColP[rh][0][kt * 32 + (lg >> 1) * 16 + l16] = x;
    }
  };

  // ---- waves 0-3: scores of item j from sColP (group mean, max-pool inside the slice clipped
  // to the prefix [0, L - w), unpooled scores, slice-edge column sums); thread = (key, head half)
  auto col = [&](bool snap, int g, int kl) -> float {
    if (!snap) return sColP[0][0][kl] + sColP[1][0][kl];
    if (NTH == 1) return sColP[g >> 1][g & 1][kl];
    if (NTH == 2) return sColP[g][0][kl];
    return sColP[0][0][kl] + sColP[1][0][kl];
  };
  auto store = [&](const PipeRef& j) {
    int tid = threadIdx.x;   // opaque per call: no per-thread store address is kept across the loop
    asm volatile("" : "+v"(tid));
    const bool snap = P.layer[j.slot].rule == RKV_SNAPKV;
    const int cbase = j.slice * kSlice, npre = L - w, ph = P.pool_half;
    float* Srow = P.S + (size_t)j.job * L;
    const float NEG_INF = -__builtin_inff();
    if (snap && NTH == 1 && G == 4 && ph == 3) {
      // the common case: four query heads, one row tile each (heads 2h, 2h + 1 in row half h),
      // 7-wide pool; thread = (key, row half)
      const int kl = tid >> 1, h = tid & 1, kk = cbase + kl;
      const float* c0 = sColP[h][0];
      const float* c1 = sColP[h][1];
      // pool window [lo, hi] inside the slice and the prefix; it holds kl whenever the pooled
      // score is used (kk < L - w).  Clamping a neighbour into the window repeats a member, which
      // leaves the maximum unchanged, so all fourteen reads are unconditional (no branches, one
      // wait); for window keys (hi < kl) the range degenerates to [lo, lo] and the result is unused
      const int lo = max(kk - 3, cbase) - cbase;
      const int hi = max(min(min(kk + 3, cbase + kSlice - 1), npre - 1) - cbase, lo);
      float a[7], b[7];
#pragma unroll
      for (int u = 0; u < 7; ++u) {
        const int qc = min(max(kl + u - 3, lo), hi);
        a[u] = c0[qc];
        b[u] = c1[qc];
      }
      float m0 = a[0], m1 = b[0];
#pragma unroll
      for (int u = 1; u < 7; ++u) {
        m0 = fmaxf(m0, a[u]);
        m1 = fmaxf(m1, b[u]);
      }
      float su = c0[kl] + c1[kl], sc = m0 + m1;
      su += dppf<0xB1>(su);   // quad_perm [1,0,3,2]: the other head half's sum (lane ^ 1)
      sc += dppf<0xB1>(sc);
      if (h == 0 && kk < L) {
        su *= inv_g;
        Srow[kk] = kk < npre ? sc * inv_g : su;
        if (P.want_unpooled) P.Su[(size_t)j.job * L + kk] = su;
      }
      if (tid < 48) {   // slice-edge column sums: head tid / 12, offsets 0..5 and 122..127
        const int g = tid / 12, o = tid - 12 * g;
        const int kl2 = o < 6 ? o : kSlice - 12 + o;
        P.edge[((size_t)j.job * nsl + j.slice) * 48 + tid] = (cbase + kl2 < L) ? sColP[g >> 1][g & 1][kl2] : 0.f;
      }
    } else if (snap) {
      const int kl = tid >> 1, kk = cbase + kl;
      const int g0 = (tid & 1) * ((G + 1) >> 1), g1 = min(G, g0 + ((G + 1) >> 1));
      float su = 0.f, sc = 0.f;
      if (kk < L) {
        const int lo = max(kk - ph, cbase) - cbase, hi = min(min(kk + ph, cbase + kSlice - 1), npre - 1) - cbase;
        for (int g = g0; g < g1; ++g) {
          su += col(true, g, kl);
          float m = NEG_INF;
          for (int u = lo; u <= hi; ++u) m = fmaxf(m, col(true, g, u));
          sc += m;
        }
      }
      su += dppf<0xB1>(su);   // quad_perm [1,0,3,2]: the other head half's sum (lane ^ 1)
      sc += dppf<0xB1>(sc);
      if ((tid & 1) == 0 && kk < L) {
        su *= inv_g;
        Srow[kk] = kk < npre ? sc * inv_g : su;
        if (P.want_unpooled) P.Su[(size_t)j.job * L + kk] = su;
      }
      if (ph > 0) {
        const int E = 4 * ph, twoP = 2 * ph;
        float* ed = P.edge + ((size_t)j.job * nsl + j.slice) * G * E;
        for (int e = tid; e < G * E; e += 256) {
          const int g = e / E, o = e - g * E;
          const int kl2 = o < twoP ? o : kSlice - twoP + (o - twoP);
          ed[e] = (cbase + kl2 < L) ? col(true, g, kl2) : 0.f;
        }
      }
    } else if (tid < kSlice && cbase + tid < L) {
      Srow[cbase + tid] = col(false, 0, tid) * inv_g;
    }
  };

  // ---- normalisers, two levels (waves 0-3).  Level 1: the workgroup scoring slice g gs of a job
  // sums the row sums of slices [g gs, g gs + gs) into partial g; level 2: every workgroup sums
  // the job's ng partials.  Both read one value per (row, slice or group) with the same mapping:
  // wave wv takes rows 32 wv + [0, 32), lane l reads rows 32 wv + 16 hh + 4 (l / 16) + [0, 4)
  // (hh = 0, 1) of slice or group l % 16, as 16-byte loads that bypass the non-coherent cache;
  // the buffer's record count makes reads past the last slice or group return 0.  A batch with a
  // value not stored yet (NaN) is read again as a whole.
  const int gs = (nsl + kPipeGroups - 1) / kPipeGroups, ng = (nsl + gs - 1) / gs;
  f32x4v l1x[2], l2x[2];
  auto sum_off = [&]() {
    // lane offset from an opaque copy of the thread index: no address is kept across the loop
    int tv = threadIdx.x;
    asm volatile("" : "+v"(tv));
    return ((tv & 15) * R + 32 * (tv >> 6) + 4 * ((tv & 63) >> 4)) * 4;
  };
  auto load_l1 = [&](const PipeRef& j) {
    const int s0 = (j.slice / gs) * gs, ns = min(gs, nsl - s0);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(P.stats + ((size_t)j.job * nsl + s0) * R), (short)0, ns * R * 4, 0x00020000);
    const int off = sum_off();
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)   // cache policy 16: sc1 (coherent at device scope)
      l1x[hh] = __builtin_bit_cast(f32x4v, __builtin_amdgcn_raw_buffer_load_b128(rs, off + hh * 64, 0, 16));
  };
  auto load_l2 = [&](int job) {
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(P.part + (size_t)job * kPipeGroups * R), (short)0, ng * R * 4, 0x00020000);
    const int off = sum_off();
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
      l2x[hh] = __builtin_bit_cast(f32x4v, __builtin_amdgcn_raw_buffer_load_b128(rs, off + hh * 64, 0, 16));
  };
  // reduce-scatter of a lane's 8 values over the 16 lanes of its row group: lanes l and l ^ 1 end
  // with the sum of row 32 wv + 4 (l / 16) + bit3(l) + 2 bit2(l) + 16 bit1(l)
  auto reduce8 = [&](const f32x4v (&x)[2]) -> float {
    float v[8];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int i = 0; i < 4; ++i) v[4 * hh + i] = x[hh][i];
    dpp_halve<0x128, 8, 8>(v, (lane >> 3) & 1);   // row_ror:8           -> lane l ^ 8
    dpp_halve<0x141, 4, 8>(v, (lane >> 2) & 1);   // row_half_mirror     -> 7 - l within 8
    dpp_halve<0x4E, 2, 8>(v, (lane >> 1) & 1);    // quad_perm [2,3,0,1] -> l ^ 2
    dpp_halve<0xB1, 1, 8>(v, 0);                  // quad_perm [1,0,3,2] -> l ^ 1
    return v[0];
  };
  const int my_row = 32 * wv + 4 * lg + 2 * ((l16 >> 2) & 1) + ((l16 >> 3) & 1) + 16 * ((l16 >> 1) & 1);
  // a sum over a batch, re-read (after a short sleep) while a value in it is not stored yet; a
  // wait that times out sets status bit 0 and stops this wave's waits
  auto settled = [&](f32x4v (&x)[2], auto&& reload) -> float {
    uint32_t it = 0;
    while (true) {
      const float z = reduce8(x);
      if (__builtin_amdgcn_ballot_w64(z != z) == 0 || gave_up) return z;
      if (++it > kSpinLimit) {
        if (lane == 0) atomicOr(status, 1u);
        gave_up = true;   // report once, then stop waiting in this workgroup
        return z;
      }
      __builtin_amdgcn_s_sleep(1);
      reload();
      wait_vmcnt<0>();
    }
  };
  auto take_l1 = [&](const PipeRef& j) {
    const float z = settled(l1x, [&] { load_l1(j); });
    if ((l16 & 1) == 0)
      __hip_atomic_store(P.part + ((size_t)j.job * kPipeGroups + j.slice / gs) * R + my_row, z, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  };
  auto take_l2 = [&](const PipeRef& j) {
    const float z = settled(l2x, [&] { load_l2(j.job); });
    if (z == __builtin_inff() && (l16 & 1) == 0) {
      // a key far above the row's reference: the job is rescored exactly before selection
      atomicOr(status, RKV_STATUS_REPAIRED);
      atomicOr(P.counters + (size_t)kCounterStride * (1 + j.job) + 1, 1u);
    }
    // z >= 1 for every valid row (the reference key contributes 1); padding rows have z = 0, and
    // a row left NaN after a time-out gets 0
    if ((l16 & 1) == 0) sAlpha[my_row] = z > 0.f && z < __builtin_inff() ? __builtin_amdgcn_rcpf(z) : 0.f;
  };

  f32x4v e0[4][2], e1[4][2], e2[4][2], e3[4][2];
  PipeRef ja = pipe_item(first, nsl, B, Hkv);   // item t
  PipeRef j1 = ja, j2 = ja, j3 = ja;              // items t - 1, t - 2, t - 3
  if (wv >= 4) {
    issue_dma(ja, 0);
    if (T > 1) {
      PipeRef jn = ja;
      pipe_advance(jn, dj, ds, nsl, B, Hkv);
      issue_dma(jn, 1);
    }
  } else {
    // every register the loop reads is defined (values unused)
    load_l1(ja);
    load_l2(min(ja.job, n_jobs - 1));
  }

  auto iteration = [&](int t, f32x4v (&ea)[4][2], f32x4v (&eb)[4][2]) {
    const bool doA = t < T, doB = t >= 3 && t - 3 < T;
    // this workgroup sums the group of item t - 1 (it scores the group's first slice)
    const bool sums = t >= 1 && t - 1 < T && j1.slice % gs == 0;
    // No barrier here: the buffers this iteration reads were filled and handed on before B1.5 of
    // iteration t - 1 (DMA of item t), B2 of t - 1 (sStat, sAlpha free again), and the score
    // stores of iteration t - 1 read the other sColP buffer.  A wave may so start phase A while
    // another wave of its SIMD is still issuing DMA.  The first iteration waits for the two
    // DMAs issued before the loop.
    if (t == 0) {
      wait_vmcnt<0>();
      lds_barrier();
    }
    sColP = sColPb[t & 1];
    // both phases run in every iteration (on stale data at the ends of the pipeline, with their
    // results unused), so each register set is redefined unconditionally
    if (!SHORT || doA) phase_a(ja, t & 1, ea);
    // MID: everything this wave issued in earlier iterations has completed (the partials of item
    // t - 3's job, the DMA of item t + 1)
    wait_vmcnt<0>();
    if (wv < 4) {
      if (doB) take_l2(j3);
      if (sums) load_l1(j1);   // item t - 1's row sums, stored at B1.5 of iteration t - 1
    }
    lds_barrier();   // B1.5: every wave's phase A is done (sStat complete, buffer t % 2 free)
    // wave 0: item t's row sums (the summing workgroup checks for sums not stored yet)
    if (wv == 0 && doA) {
      float2 o;
      o.x = sStat[0][2 * lane] + sStat[1][2 * lane] + sStat[2][2 * lane] + sStat[3][2 * lane];
      o.y = sStat[0][2 * lane + 1] + sStat[1][2 * lane + 1] + sStat[2][2 * lane + 1] + sStat[3][2 * lane + 1];
      store_coherent2(P.stats + ((size_t)ja.job * nsl + ja.slice) * R + 2 * lane, o.x, o.y);
    }
    if (!SHORT || doB) phase_b(j3, eb);
    lds_barrier();   // B2: sColP complete
    if (wv < 4) {
      if (sums) {
        // the group's row sums loaded at MID (wave 0's row-sum store may still be in flight)
        if (wv == 0 && doA) wait_vmcnt<1>();
        else wait_vmcnt<0>();
        take_l1(j1);
      }
      if (doB) store(j3);
      // the partials of item t - 2's job (stored at the end of iteration t - 1), consumed at the
      // next MID; loaded in every iteration so that the registers have one definition (the job
      // is clamped where the item lies outside the pipeline)
      load_l2(min(j2.job, n_jobs - 1));
    } else if (t + 2 < T) {
      PipeRef jn = ja;
      pipe_advance(jn, dj, ds, nsl, B, Hkv);
      pipe_advance(jn, dj, ds, nsl, B, Hkv);
      issue_dma(jn, t & 1);
    }
    j3 = j2;
    j2 = j1;
    j1 = ja;
    pipe_advance(ja, dj, ds, nsl, B, Hkv);
  };

  // T + 3 iterations drain the pipeline; the count is padded to a multiple of four (the padding
  // iterations store nothing) so that the unrolled body has a single exit at its end.  Item t's
  // exponentials live in set t % 4 from iteration t to t + 3.
  const int n_iter = (T + 3 + 3) & ~3;
#pragma unroll 1
  for (int t = 0; t < n_iter; t += 4) {
    iteration(t, e0, e1);
    iteration(t + 1, e1, e2);
    iteration(t + 2, e2, e3);
    iteration(t + 3, e3, e0);
  }
}

// Ranking key of a score: its bit pattern, whose unsigned order is the numeric order for the
// non-negative scores the scoring kernels produce.  Patterns with the sign bit set (which no
// valid score has) rank as +0, so the radix passes, which look at bits 0-30 only, and the
// comparisons against the k-th key agree for every input and the compaction never writes more
// than k positions.
__device__ __forceinline__ uint32_t rank_bits(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u >> 31) ? 0u : u;
}

// ---------------------------------------------------------------------------------------------
// Exact rescoring of one window-scored job (the repair path).  The window scoring kernels take
// their exponentials against a fixed per-row reference; a row with a key far above it overflows
// the row sum, and the kernel flags the job (word 1 of the job's counter line).  The selection
// workgroup of a flagged job recomputes the job's scores here, in plain fp32 arithmetic with a
// running maximum per row (no reference, so nothing overflows), before it ranks them:
//   pass 1: per window row r, m_r = max_j x_rj and s_r = sum_j exp2(x_rj - m_r) over its visible
//           keys, x = q.k log2(e)/sqrt(d) (thread = (row, key lane); lanes combined via LDS);
//   pass 2: per key j, A_g[j] = sum over head g's rows of exp2(x_rj - m_r) / s_r, in chunks of
//           blockDim keys that include the pool halo; S gets the pooled (SnapKV prefix) or plain
//           group mean, Su the plain group mean, as the scoring kernels store them.
// It is slow (two passes of scalar FMAs over the job) and only runs for flagged jobs; inlined,
// with the query rows read from LDS, so the selection kernels need no stack.  Needs
// G * w <= kRepairRows (256, every window-scored layout), blockDim >= kRepairRows and kRepairLds
// bytes of LDS at `lds`.
// ---------------------------------------------------------------------------------------------
constexpr int kRepairRows = kMaxRowTiles * 32;   // G * w of the window-scored layouts
constexpr int kRepairKeyLanes = 4;               // blockDim / kRepairRows at most
constexpr int kRepairLds = (kRepairRows * kHeadDim * 2) + 4 * (2 * kRepairRows + 2 * kRepairKeyLanes * kRepairRows + 8 * 1024);
static_assert(kRepairLds <= kSelectLds, "the repair runs in the selection kernels' dynamic LDS");

__device__ __forceinline__ void rescore_exact(const uint16_t* qjob, const uint16_t* khead, float* S, float* Su, int L,
                                           int w, int G, int ph, int snap, float sl2, float* lds) {
  const int T = blockDim.x, tid = threadIdx.x;
  const int R = G * w;
  uint32_t* sQ = reinterpret_cast<uint32_t*>(lds);   // [128][64] bf16 pairs of the job's query rows
  float* sM = lds + kRepairRows * kHeadDim / 2;        // [128] row maxima (log2 units)
  float* sR = sM + kRepairRows;                        // [128] reciprocal row sums
  float* sPm = sR + kRepairRows;                       // [key lanes][128] partial maxima
  float* sPs = sPm + kRepairKeyLanes * kRepairRows;    // [key lanes][128] partial sums
  float* sA = sPs + kRepairKeyLanes * kRepairRows;     // [G][T] column sums of a chunk
  const float NEG_INF = -__builtin_inff();
  for (int e = tid; e < kRepairRows * kHeadDim / 2; e += T)
    sQ[e] = (e >> 6) < R ? reinterpret_cast<const uint32_t*>(qjob)[e] : 0u;
  __syncthreads();
  // ---- pass 1
  const int nkl = T / kRepairRows, row = tid % kRepairRows, kl = tid / kRepairRows;
  {
    float m = NEG_INF, sum = 0.f;
    if (row < R) {
      const int last = L - w + row % w;   // the row's own position
      const u32x4* qr = reinterpret_cast<const u32x4*>(sQ + row * 64);
      for (int j = kl; j <= last; j += nkl) {
        const u32x4* kr = reinterpret_cast<const u32x4*>(khead + (size_t)j * kHeadDim);
        float z = 0.f;
#pragma unroll 4
        for (int c = 0; c < 16; ++c) {
          const u32x4 kv = kr[c], qv = qr[c];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            z = fmaf(__uint_as_float(qv[u] << 16), __uint_as_float(kv[u] << 16), z);
            z = fmaf(__uint_as_float(qv[u] & 0xffff0000u), __uint_as_float(kv[u] & 0xffff0000u), z);
          }
        }
        const float x = z * sl2;
        if (x > m) {
          sum = sum * __builtin_amdgcn_exp2f(m - x) + 1.f;
          m = x;
        } else {
          sum += __builtin_amdgcn_exp2f(x - m);
        }
      }
    }
    sPm[kl * kRepairRows + row] = m;
    sPs[kl * kRepairRows + row] = sum;
  }
  __syncthreads();
  if (tid < kRepairRows) {
    float m = NEG_INF, sum = 0.f;
    for (int k = 0; k < nkl; ++k) {
      const float pm = sPm[k * kRepairRows + tid], ps = sPs[k * kRepairRows + tid];
      if (!(ps > 0.f)) continue;
      if (!(sum > 0.f)) {
        m = pm;
        sum = ps;
      } else {
        const float M = fmaxf(m, pm);
        sum = sum * __builtin_amdgcn_exp2f(m - M) + ps * __builtin_amdgcn_exp2f(pm - M);
        m = M;
      }
    }
    sM[tid] = m;
    sR[tid] = sum > 0.f ? 1.f / sum : 0.f;
  }
  __syncthreads();
  // ---- pass 2
  const int core = T - 2 * ph, npre = L - w;
  const float inv_g = 1.f / (float)G;
  for (int c0 = 0; c0 < L; c0 += core) {
    const int j = c0 - ph + tid;
    const bool valid = j >= 0 && j < L;
    // the key row is re-read per window row (L2 hits) so that no 64-register copy is live
    const u32x4* kr = reinterpret_cast<const u32x4*>(khead + (size_t)(valid ? j : 0) * kHeadDim);
    for (int g = 0; g < G; ++g) {
      float acc = 0.f;
      if (valid) {
        for (int ii = 0; ii < w; ++ii) {
          if (j > L - w + ii) continue;   // row ii of the window does not see key j
          const int r = g * w + ii;
          float z = 0.f;
          const u32x4* qr = reinterpret_cast<const u32x4*>(sQ + r * 64);
#pragma unroll 4
          for (int c = 0; c < 16; ++c) {
            const u32x4 qv = qr[c], kv = kr[c];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              z = fmaf(__uint_as_float(qv[u] << 16), __uint_as_float(kv[u] << 16), z);
              z = fmaf(__uint_as_float(qv[u] & 0xffff0000u), __uint_as_float(kv[u] & 0xffff0000u), z);
            }
          }
          acc += __builtin_amdgcn_exp2f(z * sl2 - sM[r]) * sR[r];
        }
      }
      sA[g * T + tid] = acc;
    }
    __syncthreads();
    if (tid >= ph && tid < ph + core && valid) {
      float su = 0.f, sc = 0.f;
      for (int g = 0; g < G; ++g) su += sA[g * T + tid];
      if (snap && j < npre) {
        const int lo = max(j - ph, 0), hi = min(j + ph, npre - 1);
        for (int g = 0; g < G; ++g) {
          float mx = NEG_INF;
          for (int t = lo; t <= hi; ++t) mx = fmaxf(mx, sA[g * T + tid + (t - j)]);
          sc += mx;
        }
        S[j] = sc * inv_g;
      } else {
        S[j] = su * inv_g;
      }
      Su[j] = su * inv_g;
    }
    __syncthreads();
  }
  __threadfence();
  __syncthreads();
}

// ---------------------------------------------------------------------------------------------
// Selection: one workgroup per job.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void select_kernel(const PrefillLaunch P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = wave_id();
  const int Hkv = P.n_kv_heads, B = P.batch, L = P.seq_len, w = P.window, G = P.group, NC = P.n_slices;
  const int job = blockIdx.x;
  const int h = job % Hkv, s = (job / Hkv) % B, slot = job / (Hkv * B);
  const PrefillLayer& ly = P.layer[P.slot_layer[slot]];
  const int bh = s * Hkv + h;
  const bool snap = ly.rule == RKV_SNAPKV;
  const float NEG_INF = -__builtin_inff();

  constexpr int kSelFixed = kHistBins * 4 + 64;
  int* sHist = reinterpret_cast<int*>(smem);
  int* sScan = sHist + kHistBins;          // 2 * kWaves ints
  int* sSel = sScan + 8;                   // 2 ints
  float* sCache = reinterpret_cast<float*>(smem + kSelFixed);
  const int cache_cap = (kSelectLds - kSelFixed) / 4;
  float* Srow = P.S + (size_t)job * L;
  const int n_score = ly.all ? (snap ? L - w : L) : ly.cand_end;
  const int ph = P.pool_half, E = 4 * ph, twoP = 2 * ph;
  // a window-scored job flagged by the pipelined kernel is rescored exactly first; its scores
  // are then complete (no slice-border pool repair)
  const bool repaired =
      slot < P.n_window &&
      __hip_atomic_load(P.counters + (size_t)kCounterStride * (1 + job) + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
  if (repaired)
    rescore_exact(ly.q + (size_t)(s * P.n_q_heads + h * G) * w * kHeadDim, ly.k + (size_t)bh * L * kHeadDim, Srow,
                  P.Su + (size_t)job * L, L, w, G, ph, snap ? 1 : 0, P.scale_log2, reinterpret_cast<float*>(smem));
  const bool fix = snap && ph > 0 && n_score > 0 && NC > 1 && !repaired;
  const int n_edge = fix ? NC * G * E : 0;
  const bool cached = n_score + n_edge <= cache_cap;
  float* sEdge = sCache + n_score;
  const float* Erow = P.edge + (size_t)job * NC * G * E;
  if (cached) {   // eight loads in flight per thread
    for (int j0 = tid; j0 < n_score + n_edge; j0 += kThreads * 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kThreads;
        v[u] = j < n_score ? Srow[j] : (j < n_score + n_edge ? Erow[j - n_score] : 0.f);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kThreads;
        if (j < n_score + n_edge) sCache[j] = v[u];   // sEdge == sCache + n_score
      }
    }
  }
  lds_barrier();
  // SnapKV: redo the pooled score of positions within pool_half of an interior slice border
  if (fix) {
    const int npre = L - w;
    for (int e = tid; e < (NC - 1) * twoP; e += kThreads) {
      const int cb = 1 + e / twoP, o = e - (e / twoP) * twoP;
      const int bnd = cb * kSlice;
      const int j = bnd - ph + o;
      if (j < 0 || j >= npre || j >= n_score) continue;
      // slice cb-1 holds keys [bnd-2P, bnd) at offsets [2P, 4P); slice cb keys [bnd, bnd+2P) at [0, 2P)
      const int left = (cb - 1) * G * E, right = cb * G * E;
      const int lo = max(j - ph, 0), hi = min(j + ph, npre - 1);
      float sc = 0.f;
      for (int g = 0; g < G; ++g) {
        float m = NEG_INF;
        for (int t = lo; t <= hi; ++t) {
          const int ei = (t < bnd) ? left + g * E + twoP + (t - (bnd - twoP)) : right + g * E + (t - bnd);
          m = fmaxf(m, cached ? sEdge[ei] : Erow[ei]);
        }
        sc += m;
      }
      if (cached) sCache[j] = sc / (float)G;
      else Srow[j] = sc / (float)G;
    }
  }
  lds_barrier();
  auto get = [&](int j) -> float { return cached ? sCache[j] : Srow[j]; };
  if (ly.score) {
    float* so = ly.score + (size_t)bh * L;
    for (int j = tid; j < n_score; j += kThreads) so[j] = get(j);
  }
  int32_t* idx = ly.idx + (size_t)bh * ly.n_keep;
  if (ly.all) {
    for (int m = tid; m < ly.n_keep; m += kThreads) idx[m] = m;
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
        lds_barrier();
        for (int j = tid; j < n; j += kThreads) {
          const uint32_t x = rank_bits(get(j));
          if ((x & pmask) == prefix) atomicAdd(&sHist[(x >> shift) & (nb - 1)], 1);
        }
        lds_barrier();
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
        lds_barrier();
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
        lds_barrier();
        prefix |= (uint32_t)sSel[0] << shift;
        pmask |= (uint32_t)(nb - 1) << shift;
        kk = sSel[1];
        lds_barrier();
      }
      const uint32_t tau = prefix;
      const int need = kk;  // ties at tau taken in position order
      // ordered compaction: wave wv owns a contiguous key range; within it, 64 keys at a time,
      // ballots give each taken key its rank among the greater / equal keys before it
      const int per_w = ((n + kWaves - 1) / kWaves + 63) & ~63;
      const int w0 = min(n, wv * per_w), w1 = min(n, w0 + per_w);
      const uint64_t lt = (1ull << lane) - 1ull;
      int cg = 0, ce = 0;
      for (int j0 = w0; j0 < w1; j0 += 64) {
        const int j = j0 + lane;
        const uint32_t x = j < w1 ? rank_bits(get(j)) : 0u;
        cg += __popcll(__ballot(j < w1 && x > tau));
        ce += __popcll(__ballot(j < w1 && x == tau));
      }
      if (lane == 0) {
        sScan[2 * wv] = cg;
        sScan[2 * wv + 1] = ce;
      }
      lds_barrier();
      int bg = 0, be = 0;   // greater / equal keys before this wave's range
      for (int i = 0; i < wv; ++i) {
        bg += sScan[2 * i];
        be += sScan[2 * i + 1];
      }
      for (int j0 = w0; j0 < w1; j0 += 64) {
        const int j = j0 + lane;
        const uint32_t x = j < w1 ? rank_bits(get(j)) : 0u;
        const bool gt = j < w1 && x > tau, eq = j < w1 && x == tau;
        const uint64_t mg = __ballot(gt), me = __ballot(eq);
        const int rg = bg + __popcll(mg & lt), re = be + __popcll(me & lt);
        if (gt) idx[rg + min(re, need)] = j;
        else if (eq && re < need) idx[rg + re] = j;
        bg += __popcll(mg);
        be += __popcll(me);
      }
    }
    const int nf = ly.forced_hi - ly.forced_lo;
    for (int t = tid; t < nf; t += kThreads) idx[k + t] = ly.forced_lo + t;
  }
  if (ly.acc) {
    // scores of the retained positions (they seed decode-phase accumulation)
    lds_barrier();
    const float* accsrc = snap ? P.Su + (size_t)job * L : Srow;
    float* acc = ly.acc + (size_t)bh * ly.n_keep;
    for (int m = tid; m < ly.n_keep; m += kThreads) acc[m] = accsrc[idx[m]];
  }
}

// Selection with every candidate score held in registers (kSelRegs = 8, 16 or 32 per thread, 1024
// threads: prompts of up to 8K, 16K or 32K keys):
// wave wv owns the contiguous key range [w0, w1); its lane l holds keys w0 + 64 i + l.  Dynamic
// LDS holds the job's slice-edge column sums and the repaired scores next to slice borders
// (with their per-head pool maxima).
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
static_assert(kSelWaves <= 16, "wave prefixes are summed over one 16-lane DPP row");
constexpr int kSelRegsMax = 32;                              // scores per thread, at most
constexpr int kSelRegsMaxKeys = kSelRegsMax * kSelThreads;   // 32K keys

template <int kSelRegs>
__global__ __launch_bounds__(kSelThreads) void select_regs_kernel(const PrefillLaunch P) {
  // dynamic LDS: [n_edge] edges, [n_fix] repaired scores (or the exact rescoring's staging)
  extern __shared__ __attribute__((aligned(16))) float sDyn[];
  __shared__ int sHist[2][kHistBins];   // pass p uses buffer p % 2
  __shared__ int sScan[2 * kSelWaves];
  __shared__ int sSel[2][2];            // likewise
  __shared__ uint32_t sRange[2][kSelWaves];   // per-wave smallest and largest ranking key
  const int tid = threadIdx.x, lane = tid & 63, wv = wave_id(), l16 = lane & 15;
  const int Hkv = P.n_kv_heads, B = P.batch, L = P.seq_len, w = P.window, G = P.group, NC = P.n_slices;
  const int job = blockIdx.x;
  const int h = job % Hkv, s = (job / Hkv) % B, slot = job / (Hkv * B);
  const PrefillLayer& ly = P.layer[P.slot_layer[slot]];
  const int bh = s * Hkv + h;
  const bool snap = ly.rule == RKV_SNAPKV;
  const float NEG_INF = -__builtin_inff();
  const float inv_g = 1.f / (float)G;
  const float* Srow = P.S + (size_t)job * L;
  const int n = ly.all ? (snap ? L - w : L) : ly.cand_end;   // candidate (and reported) positions
  const int ph = P.pool_half, E = 4 * ph, twoP = 2 * ph;
  // the repair flag, the candidate scores and the slice-edge sums are requested together (one
  // round trip); a window-scored job flagged by the pipelined kernel (rare) is then rescored
  // exactly and its scores read again, complete (no slice-border pool repair)
  const uint32_t flag =
      slot < P.n_window
          ? __hip_atomic_load(P.counters + (size_t)kCounterStride * (1 + job) + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
          : 0u;
  const bool fix0 = snap && ph > 0 && n > 0 && NC > 1;
  const int n_edge0 = fix0 ? NC * G * E : 0;

  // ---- candidate scores into registers, slice-edge sums into LDS.  The waves' ranges are cut
  // from the prompt length, a kernel argument, so that the score loads do not wait for the
  // layer-table lookups that give the candidate count n; positions from n on are not candidates
  const int per_w = ((L + kSelWaves - 1) / kSelWaves + 63) & ~63;
  const int w0 = wv * per_w, wL = min(L, w0 + per_w), w1 = min(n, w0 + per_w);
  float x[kSelRegs];
#pragma unroll
  for (int i = 0; i < kSelRegs; ++i) {
    const int j = w0 + 64 * i + lane;
    x[i] = j < wL ? Srow[j] : 0.f;
  }
  if (fix0) {
    const float* Erow = P.edge + (size_t)job * NC * G * E;
    for (int e0 = tid; e0 < n_edge0; e0 += kSelThreads * 4) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = e0 + u * kSelThreads < n_edge0 ? Erow[e0 + u * kSelThreads] : 0.f;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (e0 + u * kSelThreads < n_edge0) sDyn[e0 + u * kSelThreads] = v[u];
    }
  }
  loads_done();
  const bool repaired = flag != 0u;
  if (repaired) {
    __syncthreads();   // the edge sums written above are done before the rescoring reuses that LDS
    rescore_exact(ly.q + (size_t)(s * P.n_q_heads + h * G) * w * kHeadDim, ly.k + (size_t)bh * L * kHeadDim,
                  P.S + (size_t)job * L, P.Su + (size_t)job * L, L, w, G, ph, snap ? 1 : 0, P.scale_log2, sDyn);
    // the rescored values, past any copy the loads above left in the non-coherent cache
#pragma unroll
    for (int i = 0; i < kSelRegs; ++i) {
      const int j = w0 + 64 * i + lane;
      x[i] = j < w1 ? __hip_atomic_load(Srow + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0.f;
    }
    loads_done();
  }
  const bool fix = fix0 && !repaired;
  const int n_edge = fix ? n_edge0 : 0, n_fix = fix ? (NC - 1) * twoP : 0;
  float* sEdge = sDyn;
  float* sFix = sDyn + n_edge;
  if (fix) {
    lds_barrier();
    // SnapKV: redo the pooled score of positions within pool_half of an interior slice border;
    // slice cb-1 holds keys [bnd-2P, bnd) at edge offsets [2P, 4P), slice cb keys [bnd, bnd+2P) at [0, 2P)
    // one thread per position: the pool maximum of every head, summed in head order
    const int npre = L - w;
    if (G == 4 && ph == 3) {
      // the common layout: four heads, 7-wide pool, every read issued at once (neighbours clamped
      // into the pool window repeat a member, which leaves the maximum unchanged)
      for (int e = tid; e < n_fix; e += kSelThreads) {
        const int cb = 1 + e / 6, o = e - (cb - 1) * 6;
        const int bnd = cb * kSlice, j = bnd - 3 + o;
        const bool ok = j >= 0 && j < npre && j < n;
        const int lo = ok ? max(j - 3, 0) : bnd, hi = ok ? min(j + 3, npre - 1) : bnd;
        float sc = 0.f;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int left = (cb - 1) * 4 * 12 + g * 12 + 6 - (bnd - 6), right = cb * 4 * 12 + g * 12 - bnd;
          float m = NEG_INF;
#pragma unroll
          for (int u = 0; u < 7; ++u) {
            const int t = min(max(j - 3 + u, lo), hi);
            m = fmaxf(m, sEdge[t < bnd ? left + t : right + t]);
          }
          sc += m;
        }
        sFix[e] = ok ? sc * inv_g : 0.f;
      }
    } else {
      for (int e = tid; e < n_fix; e += kSelThreads) {
        const int cb = 1 + e / twoP, o = e - (cb - 1) * twoP;
        const int bnd = cb * kSlice, j = bnd - ph + o;
        float sc = 0.f;
        if (j >= 0 && j < npre && j < n) {
          const int lo = max(j - ph, 0), hi = min(j + ph, npre - 1);
          for (int g = 0; g < G; ++g) {
            const int left = (cb - 1) * G * E + g * E + twoP - (bnd - twoP), right = cb * G * E + g * E - bnd;
            float m = NEG_INF;
            for (int t = lo; t <= hi; ++t) m = fmaxf(m, sEdge[t < bnd ? left + t : right + t]);
            sc += m;
          }
        }
        sFix[e] = sc * inv_g;
      }
    }
    lds_barrier();
#pragma unroll
    for (int i = 0; i < kSelRegs; ++i) {
      const int j = w0 + 64 * i + lane;
      const int cb = (j + ph) / kSlice, o = j + ph - cb * kSlice;
      if (j < w1 && j < npre && cb >= 1 && cb < NC && o < twoP) x[i] = sFix[(cb - 1) * twoP + o];
    }
  }
  if (ly.score) {
    float* so = ly.score + (size_t)bh * L;
#pragma unroll
    for (int i = 0; i < kSelRegs; ++i) {
      const int j = w0 + 64 * i + lane;
      if (j < w1) so[j] = x[i];
    }
  }
  int32_t* idx = ly.idx + (size_t)bh * ly.n_keep;
  if (ly.all) {
    for (int m = tid; m < ly.n_keep; m += kSelThreads) idx[m] = m;
  } else {
    const int k = ly.k_sel;
    if (k > 0) {
      // k-th largest candidate score: radix passes over the ranking keys (scores are >= 0, so the
      // unsigned order of their bit patterns is the numeric order) taken relative to the
      // smallest candidate key, d = u - umin: the first pass bins the top 11 bits of the span
      // [0, umax - umin], which spreads the candidates over its 2048 bins (the scores of a job
      // span far fewer binades than a float holds, and same-bin atomics serialise), the next
      // passes 10 bits each until every bit is resolved (at most three passes)
      uint32_t umin = 0xffffffffu, umax = 0u;
#pragma unroll
      for (int i = 0; i < kSelRegs; ++i) {
        const int j = w0 + 64 * i + lane;
        const uint32_t u = rank_bits(x[i]);
        if (j < w1) {
          umin = min(umin, u);
          umax = max(umax, u);
        }
      }
      // wave minimum and maximum: DPP inside the rows, then the four rows' results
      umin = row16_umin(umin);
      umax = row16_umax(umax);
      umin = min(min((uint32_t)__builtin_amdgcn_readlane((int)umin, 0), (uint32_t)__builtin_amdgcn_readlane((int)umin, 16)),
                 min((uint32_t)__builtin_amdgcn_readlane((int)umin, 32), (uint32_t)__builtin_amdgcn_readlane((int)umin, 48)));
      umax = max(max((uint32_t)__builtin_amdgcn_readlane((int)umax, 0), (uint32_t)__builtin_amdgcn_readlane((int)umax, 16)),
                 max((uint32_t)__builtin_amdgcn_readlane((int)umax, 32), (uint32_t)__builtin_amdgcn_readlane((int)umax, 48)));
      if (lane == 0) {
        sRange[0][wv] = umin;
        sRange[1][wv] = umax;
      }
      uint32_t prefix = 0u, pmask = 0u;
      int kk = k;
      // both histogram buffers start cleared; buffer 0 is cleared again during pass 1 (pass 0's
      // last read of it precedes pass 0's last barrier), so a pass needs three barriers
      for (int b = tid; b < 2 * kHistBins; b += kSelThreads) (&sHist[0][0])[b] = 0;
      lds_barrier();
      // the workgroup's: one read per lane (wave l16's values), a 16-lane DPP reduction
      umin = row16_umin(l16 < kSelWaves ? sRange[0][l16] : 0xffffffffu);
      umax = row16_umax(l16 < kSelWaves ? sRange[1][l16] : 0u);
      const int span_bits = 32 - __builtin_clz((umax - umin) | 1u);
      int shift = max(0, span_bits - 11);
#pragma unroll 1
      for (int pass = 0; pass < 3; ++pass) {
        if (pass > 0) {
          if (shift == 0) break;   // every bit resolved
          shift = max(0, shift - 10);
        }
        const int nb = pass == 0 ? 2048 : 1024;
        int* hist = sHist[pass & 1];
        int* sel = sSel[pass & 1];
#pragma unroll
        for (int i = 0; i < kSelRegs; ++i) {
          const int j = w0 + 64 * i + lane;
          const uint32_t d = rank_bits(x[i]) - umin;
          if (j < w1 && (d & pmask) == prefix) atomicAdd(&hist[(d >> shift) & (nb - 1)], 1);
        }
        if (pass == 1)
          for (int b = tid; b < 1024; b += kSelThreads) sHist[0][b] = 0;   // for pass 2
        lds_barrier();
        // bins in descending order: thread tid owns bins nb-1-tid*per .. (per = 2 or 1)
        const int per = nb / kSelThreads;
        int cnt = 0;
        for (int q = 0; q < per; ++q) cnt += hist[nb - 1 - (tid * per + q)];
        const int inc = wave_inclusive_scan(cnt);   // inclusive scan of cnt over the wave
        if (lane == 63) sScan[wv] = inc;
        lds_barrier();
        // plus the counts of the waves before this one: one read per lane, a 16-lane sum
        int above = inc - cnt + row16_sum(l16 < wv ? sScan[l16] : 0);
        if (kk > above && kk <= above + cnt) {
          for (int q = 0; q < per; ++q) {
            const int b = nb - 1 - (tid * per + q);
            const int hb = hist[b];
            if (kk <= above + hb) {
              sel[0] = b;
              sel[1] = kk - above;
              break;
            }
            above += hb;
          }
        }
        lds_barrier();
        // a later pass's bin field may overlap bits an earlier pass fixed: those bits of sel
        // equal the prefix's (every counted key matched it), so OR-ing them changes nothing
        prefix |= (uint32_t)sel[0] << shift;
        pmask |= (uint32_t)(nb - 1) << shift;
        kk = sel[1];
      }
      const uint32_t tau = umin + prefix;
      const int need = kk;  // ties at tau taken in position order
      // ordered compaction over the waves' contiguous ranges: ballots rank each taken key
      // among the greater / equal keys before it
      const uint64_t lt = (1ull << lane) - 1ull;
      int cg = 0, ce = 0;
#pragma unroll
      for (int i = 0; i < kSelRegs; ++i) {
        const int j = w0 + 64 * i + lane;
        const uint32_t u = rank_bits(x[i]);
        cg += __popcll(__ballot(j < w1 && u > tau));
        ce += __popcll(__ballot(j < w1 && u == tau));
      }
      if (lane == 0) {
        sScan[2 * wv] = cg;
        sScan[2 * wv + 1] = ce;
      }
      lds_barrier();
      int bg = row16_sum(l16 < wv ? sScan[2 * l16] : 0), be = row16_sum(l16 < wv ? sScan[2 * l16 + 1] : 0);
#pragma unroll
      for (int i = 0; i < kSelRegs; ++i) {
        const int j = w0 + 64 * i + lane;
        const uint32_t u = rank_bits(x[i]);
        const bool gt = j < w1 && u > tau, eq = j < w1 && u == tau;
        const uint64_t mg = __ballot(gt), me = __ballot(eq);
        const int rg = bg + __popcll(mg & lt), re = be + __popcll(me & lt);
        if (gt) idx[rg + min(re, need)] = j;
        else if (eq && re < need) idx[rg + re] = j;
        bg += __popcll(mg);
        be += __popcll(me);
      }
    }
    const int nf = ly.forced_hi - ly.forced_lo;
    for (int t = tid; t < nf; t += kSelThreads) idx[k + t] = ly.forced_lo + t;
  }
  if (ly.acc) {
    // scores of the retained positions (they seed decode-phase accumulation)
    lds_barrier();
    const float* accsrc = snap ? P.Su + (size_t)job * L : Srow;
    float* acc = ly.acc + (size_t)bh * ly.n_keep;
    for (int m = tid; m < ly.n_keep; m += kSelThreads) acc[m] = accsrc[idx[m]];
  }
}

// ---------------------------------------------------------------------------------------------
// Gather: copy the retained K / V rows, 16 lanes x 16 B per row.
// ---------------------------------------------------------------------------------------------
// Gather: the retained K and V rows, bit for bit.  Work items are (gather layer, kGatherRows
// output rows), flat over the layer's (sequence, KV head, kept row) rows, so an item never spans
// two layers and the layer is looked up once per item; thread = (row tid / 16 + 16 u, 16-byte
// piece tid % 16).  Unscored layers (StreamingLLM, Full) also write their closed-form positions
// and a zero accumulator.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void gather_kernel(const PrefillLaunch P) {
  constexpr int U = kGatherRows / 16;
  const int tid = threadIdx.x, piece = tid & 15, rsub = tid >> 4;
  const int Hkv = P.n_kv_heads, L = P.seq_len, n_gl = P.n_gather;
  const int n_items = P.gather_item0[n_gl];
  int li = 0;
  for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
    while (li + 1 < n_gl && P.gather_item0[li + 1] <= item) ++li;   // items only grow
    const PrefillLayer& ly = P.layer[P.gather_layer[li]];
    const int n_keep = ly.n_keep, rows = P.batch * Hkv * n_keep;
    const int o0 = (item - P.gather_item0[li]) * kGatherRows;
    const bool scored = ly.slot >= 0;
    int pos[U], bh[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int o = o0 + rsub + 16 * u;
      pos[u] = -1;
      bh[u] = 0;
      if (o < rows) {
        bh[u] = o / n_keep;
        const int m = o - bh[u] * n_keep;
        pos[u] = scored ? ly.idx[o] : (ly.all ? m : (m < ly.cand_end ? m : ly.forced_lo + (m - ly.cand_end)));
      }
    }
    loads_done();
    u32x4 kv[U], vv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (pos[u] >= 0) {
        const size_t src = ((size_t)bh[u] * L + pos[u]) * kHeadDim + piece * 8;
        kv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ly.k + src));
        vv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ly.v + src));
      }
    }
    loads_done();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (pos[u] >= 0) {
        const int o = o0 + rsub + 16 * u;
        const size_t dst = (size_t)o * kHeadDim + piece * 8;
        __builtin_nontemporal_store(kv[u], reinterpret_cast<u32x4*>(ly.k_out + dst));
        __builtin_nontemporal_store(vv[u], reinterpret_cast<u32x4*>(ly.v_out + dst));
        if (!scored && piece == 0) {
          ly.idx[o] = pos[u];
          if (ly.acc) ly.acc[o] = 0.f;
        }
      }
    }
  }
}

int device_cus() {
  static int cached = -1;
  if (cached < 0) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
      cus = 256;
    cached = cus;
  }
  return cached;
}

// Resident workgroups of the pipelined kernel (one per CU; the same for every NTH).
int resident_pipe_groups() {
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, score_pipe_kernel<1, false>, kPipeThreads, 0) != hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  return per_cu * device_cus();
}

// Launches one kernel that makes up a whole profiling stage; while that stage is profiled, the
// launch records the dispatch's own start and stop timestamps in the profiler's events.
template <typename... KArgs, typename... Args>
void launch_staged(int stage, void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem, hipStream_t st,
                   Args... args) {
  void *a = nullptr, *b = nullptr;
  if (profile_kernel_events(stage, &a, &b))
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)shmem, st, reinterpret_cast<hipEvent_t>(a),
                          reinterpret_cast<hipEvent_t>(b), 0u, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, shmem, st, args...);
}

}  // namespace

int launch_prefill(const PrefillLaunch& P, int row_tiles, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  // window-scored jobs (the scoring kernels below), then every scored job (selection)
  const int n_jobs = P.batch * P.n_window * P.n_kv_heads;
  const int n_sel = P.batch * P.n_scored * P.n_kv_heads;
  const int ntg = P.row_tiles_per_group;
  // the pipelined kernel takes four row tiles when a job has at most 64 slices (8192 keys) and
  // every slice of a job fits in the resident workgroups; other layouts take the window kernels
  // (window.hip), which the test hook RKV_FORCE_WINDOW=1 selects everywhere
  static const int pipe_wg = resident_pipe_groups();
  const bool pipe = n_jobs > 0 && row_tiles == 4 && P.force_window == 0 && P.n_slices <= kPipeMaxSlices &&
                    P.n_slices <= pipe_wg;
  const dim3 prep_grid(n_jobs * kPrepParts), prep_block(kPrepThreads);
  if (pipe) {
    if (ntg == 1) launch_staged(kStageZero, prepare_kernel<1>, prep_grid, prep_block, 0, st, P);
    else if (ntg == 2) launch_staged(kStageZero, prepare_kernel<2>, prep_grid, prep_block, 0, st, P);
    else launch_staged(kStageZero, prepare_kernel<4>, prep_grid, prep_block, 0, st, P);
  } else {
    // the status word is cleared even without jobs
    const int n_cnt = kCounterStride * (1 + n_jobs);
    const int blocks = std::max(1, std::min(64, (n_cnt + 255) / 256));
    launch_staged(kStageZero, reset_counters, dim3(blocks), dim3(256), 0, st, P.counters, n_cnt, (int)P.first_group);
  }
  if (n_jobs > 0) {
    if (pipe) {
      const int64_t n_items = (int64_t)n_jobs * P.n_slices;
      const int n_wg = (int)std::min<int64_t>(n_items, pipe_wg);
      // profiled, this kernel runs 10-20 % slower than in unprofiled passes (whatever event marks
      // its completion: dispatch timestamps or a marker after it), so its profiled time is an
      // upper bound; kernel traces of unprofiled passes give the undisturbed time
      const dim3 grid(n_wg), block(kPipeThreads);
      // at most kPipeShortItems items per workgroup: the form that skips the stale phases
      const bool short_run = (n_items + n_wg - 1) / n_wg <= kPipeShortItems;
      if (short_run) {
        if (ntg == 1) launch_staged(kStageScore, score_pipe_kernel<1, true>, grid, block, 0, st, P, n_wg);
        else if (ntg == 2) launch_staged(kStageScore, score_pipe_kernel<2, true>, grid, block, 0, st, P, n_wg);
        else launch_staged(kStageScore, score_pipe_kernel<4, true>, grid, block, 0, st, P, n_wg);
      } else {
        if (ntg == 1) launch_staged(kStageScore, score_pipe_kernel<1, false>, grid, block, 0, st, P, n_wg);
        else if (ntg == 2) launch_staged(kStageScore, score_pipe_kernel<2, false>, grid, block, 0, st, P, n_wg);
        else launch_staged(kStageScore, score_pipe_kernel<4, false>, grid, block, 0, st, P, n_wg);
      }
    } else {
      // longer prompts and eight row tiles: row normalisers, then column sums
      profile_mark(kStageScore, false, stream);
      const int err = launch_window(P, row_tiles, stream);
      profile_mark(kStageScore, true, stream);
      if (err) return err;
    }
  }
  if (P.n_full > 0) {
    // H2O layers with full-span accumulation: their own two passes, then the shared selection
    profile_mark(kStageScore, false, stream);
    int err = launch_fullspan(P, stream);
    profile_mark(kStageScore, true, stream);
    if (err) return err;
  }
  if (P.n_scored > P.n_window + P.n_full) {
    // TOVA layers: the last query's attention over every key, then the shared selection
    profile_mark(kStageScore, false, stream);
    int err = launch_tova(P, stream);
    profile_mark(kStageScore, true, stream);
    if (err) return err;
  }
  if (n_sel > 0) {
    static bool lds_set = false;
    if (!lds_set) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(select_kernel),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, kSelectLds);
      if (e == hipSuccess)
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(select_regs_kernel<8>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, kSelectLds);
      if (e == hipSuccess)
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(select_regs_kernel<16>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, kSelectLds);
      if (e == hipSuccess)
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(select_regs_kernel<32>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, kSelectLds);
      if (e != hipSuccess) return (int)e;
      lds_set = true;
    }
    // registers hold every candidate score when the prompt is short enough and the edge sums fit
    const size_t dyn = sizeof(float) * ((size_t)P.n_slices * P.group * 4 * P.pool_half +
                                        (size_t)(P.n_slices > 0 ? P.n_slices - 1 : 0) * 2 * P.pool_half *
                                            (1 + P.group));
    if (P.seq_len <= kSelRegsMaxKeys && dyn <= (size_t)kSelectLds - 2 * kHistBins * 4 - 256) {
      const size_t lds = std::max(dyn, (size_t)kRepairLds);
      if (P.seq_len <= 8 * kSelThreads)
        launch_staged(kStageSelect, select_regs_kernel<8>, dim3(n_sel), dim3(kSelThreads), lds, st, P);
      else if (P.seq_len <= 16 * kSelThreads)
        launch_staged(kStageSelect, select_regs_kernel<16>, dim3(n_sel), dim3(kSelThreads), lds, st, P);
      else
        launch_staged(kStageSelect, select_regs_kernel<32>, dim3(n_sel), dim3(kSelThreads), lds, st, P);
    }
    else
      launch_staged(kStageSelect, select_kernel, dim3(n_sel), dim3(kThreads), kSelectLds, st, P);
  }
  const int n_gather_items = P.n_gather > 0 ? P.gather_item0[P.n_gather] : 0;
  if (n_gather_items > 0) {
    // one workgroup per item: later workgroups' reads overlap earlier ones' writes
    const int grid = n_gather_items;
    launch_staged(kStageGather, gather_kernel, dim3(grid), dim3(kThreads), 0, st, P);
  }
  return (int)hipGetLastError();
}

}  // namespace rkv
