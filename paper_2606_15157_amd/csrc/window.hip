// Window scoring for prompts outside the pipelined kernel's range (more than 64 slices of 128
// keys per job, or eight row tiles: G * ceil(w / 32) > 4) on gfx950.  Per (sequence, layer, KV
// head) job the scores are those of the pipelined kernel (Section 2.1's SnapKV and H2O rules):
//   A[g][j] = sum_i softmax_j(Q[g,i] . K[j] / sqrt(d)), S = mean_g maxpool(A[g]) or mean_g A[g],
// computed in two passes over the keys instead of one pass with a cross-workgroup exchange:
//
// window_rows_kernel<NRT>: one workgroup per job (per part of its keys when there are few jobs:
//   the columns kernel then adds the parts' row sums), one wave per 32 window rows (R = 32 NRT
//   rows, the query rows of every head of the group, padded).  The wave's query fragments stay in
//   registers; 128-key tiles stream through two LDS buffers (LDS DMA, one tile ahead) and bf16
//   MFMA logits are taken against a fixed per-row reference c_r = max(logit with the row's own
//   key, logit with key 0), both true logits of the row; each lane sums e =
//   exp2((z - c_r) log2(e) / sqrt(d)) over its keys.  The row's log2 normaliser Lambda_r = c_r
//   log2(e)/sqrt(d) + log2(Z_r) goes to the workspace; a row whose sum overflows (a key more than
//   ~88 natural-log units above its reference) flags the job for the exact rescoring of the
//   selection kernels.  On tiles without masks the MFMAs of one half-tile run interleaved with
//   the exponentials of the other half.
// window_cols_kernel<NRT>: one workgroup per (job, 32 consecutive 128-key blocks); the job's
//   query block and normalisers sit in LDS, each of the four waves keeps its 32 keys' fragments
//   in registers (the next block's requested while the current one is scored), takes
//   p = exp2(z log2(e)/sqrt(d) - Lambda_r) over 64-row chunks (one chunk's MFMAs beside the
//   previous chunk's exponentials, also across blocks) and sums it per query head in registers;
//   the per-head column sums then give the block's pooled and unpooled scores and slice-edge
//   sums in the layout of the pipelined kernel, so the same selection (with its slice-border
//   pool repair) follows.
// Sums run in a fixed order (the only atomics set overflow flags): results are reproducible.
#include <hip/hip_runtime.h>

#include <math.h>

#include "lds_dma.h"
#include "rkv_internal.h"

namespace rkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kMaskedW = -1e30f;   // exponent of a hidden key: exp2 gives 0
constexpr int kColBlocks = 32;        // key blocks per columns workgroup

__device__ __forceinline__ bf16x8 as_bf16x8w(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int CTRL>
__device__ __forceinline__ float dpp_addw(float x) {
  return x + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}

// LDS position of 16-byte chunk `ch` of row `row` of a [rows][128] bf16 tile (XOR swizzle).
__device__ __forceinline__ int swzw(int row, int ch) { return (row * 16 + (ch ^ (row & 15))) * 8; }

// Window row r of a job: query head g = r / tpr and window index ii = r % tpr (tpr = rows per
// head in the padded layout); valid when g < G and ii < w.
struct WinRow {
  int g, ii;
  bool valid;
};
__device__ __forceinline__ WinRow win_row(int r, int tpr, int G, int w) {
  WinRow x;
  x.g = r / tpr;
  x.ii = r - x.g * tpr;
  x.valid = x.g < G && x.ii < w;
  return x;
}

template <int NRT>
__global__ __launch_bounds__(NRT * 64, 1) void window_rows_kernel(const PrefillLaunch P) {
  constexpr int R = NRT * 32, NT = NRT * 64;
  // LDS DMA of a 128-key tile: 32 instructions of 4 keys (1 KiB) each, NI per wave
  constexpr int NI = kSlice / 4 / NRT;
  static_assert(NI % 2 == 0 && NRT % 4 == 0, "instruction pairs 4 KiB apart, waves in groups of four");
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kSlice * kHeadDim];
  __shared__ float sC[R];
  const int tid = threadIdx.x, lane = tid & 63, lg = lane >> 4, l16 = lane & 15;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int L = P.seq_len, w = P.window, G = P.group, Hq = P.n_q_heads, Hkv = P.n_kv_heads, B = P.batch;
  const int tpr = P.row_tiles_per_group * 32;
  const int parts = P.window_parts, job = blockIdx.x / parts, part = blockIdx.x - job * parts;
  const int h = job % Hkv, s = (job / Hkv) % B, slot = job / (Hkv * B);
  const PrefillLayer& ly = P.layer[slot];
  const uint16_t* khead = ly.k + (size_t)(s * Hkv + h) * L * kHeadDim;
  const uint16_t* qjob = ly.q + (size_t)(s * Hq + h * G) * w * kHeadDim;   // [G][w][d]
  // this workgroup's key tiles [t0, t1) (part `part` of the job's tiles)
  const int n_tiles = (L + kSlice - 1) / kSlice;
  const int per_part = (n_tiles + parts - 1) / parts;
  const int t0 = min(n_tiles, part * per_part), t1 = min(n_tiles, t0 + per_part);

  // ---- per-row reference (every part computes the same): thread r < R takes row r (its own key and key 0, 128-d dot products)
  if (tid < R) {
    const WinRow x = win_row(tid, tpr, G, w);
    float zd = 0.f, zs = 0.f;
    if (x.valid) {
      const u32x4* qp = reinterpret_cast<const u32x4*>(qjob + (size_t)(x.g * w + x.ii) * kHeadDim);
      const u32x4* kd = reinterpret_cast<const u32x4*>(khead + (size_t)(L - w + x.ii) * kHeadDim);
      const u32x4* ks = reinterpret_cast<const u32x4*>(khead);
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const u32x4 qa = qp[c], da = kd[c], sa = ks[c];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float q0 = __uint_as_float(qa[u] << 16), q1 = __uint_as_float(qa[u] & 0xffff0000u);
          zd = fmaf(q0, __uint_as_float(da[u] << 16), zd);
          zd = fmaf(q1, __uint_as_float(da[u] & 0xffff0000u), zd);
          zs = fmaf(q0, __uint_as_float(sa[u] << 16), zs);
          zs = fmaf(q1, __uint_as_float(sa[u] & 0xffff0000u), zs);
        }
      }
    }
    sC[tid] = fmaxf(zd, zs);
  }
  // ---- the wave's query fragments: rows 32 wv + 16 rs + l16, chunk 4 st + lg
  bf16x8 qa[2][4];
#pragma unroll
  for (int rs = 0; rs < 2; ++rs) {
    const WinRow x = win_row(32 * wv + 16 * rs + l16, tpr, G, w);
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (x.valid) v = *reinterpret_cast<const u32x4*>(qjob + (size_t)(x.g * w + x.ii) * kHeadDim + 8 * (4 * st + lg));
      qa[rs][st] = as_bf16x8w(v);
    }
  }
  // Wave wv moves instructions I = (wv % 4) + 4 u + 16 (wv / 4), u = 0 .. NI - 1: keys 4 I + [0, 4)
  // of the tile, lane l filling key 4 I + l / 16 at chunk position l % 16 (the XOR swizzle of
  // swzw, so the lane's source chunk is (l % 16) ^ ((4 I + l / 16) % 16)).  I % 4 is the wave's,
  // so the lane's byte offset is the same for every instruction; instructions u and u + 1 are
  // 4 KiB apart and go as one pair.  The tile past the prompt's end repeats its last key.
  const uint32_t dma_off = (uint32_t)(lane >> 4) * 256u + (uint32_t)((lane & 15) ^ (4 * (wv & 3) + (lane >> 4))) * 16u;
  const int i0 = (wv & 3) + 16 * (wv >> 2);
  auto issue = [&](int kt, int buf) {
    const uint32_t lds0 = lds_addr(&sK[buf][0]);
    if (kt * kSlice + kSlice <= L) {
      const char* tile = reinterpret_cast<const char*>(khead + (size_t)kt * kSlice * kHeadDim);
#pragma unroll
      for (int u = 0; u < NI; u += 2) {
        const int I = i0 + 4 * u;
        dma16s_pair(tile + 1024u * I, dma_off, lds0 + 1024u * I);
      }
    } else {
#pragma unroll
      for (int u = 0; u < NI; ++u) {
        const int I = i0 + 4 * u, r = 4 * I + (lane >> 4);
        const int key = min(kt * kSlice + r, L - 1);
        dma16(khead + (size_t)key * kHeadDim + 8 * ((lane & 15) ^ (r & 15)), lds0 + 1024u * I);
      }
    }
  };
  // the first two tiles (the second stays in flight)
  if (t0 < t1) issue(t0, 0);
  if (t0 + 1 < t1) issue(t0 + 1, 1);
  __syncthreads();   // sC complete
  const float sl2 = P.scale_log2;
  float ncs[2][4], Z[2][4];
  int last[2][4];   // the row's last visible key (-1: a padding row)
#pragma unroll
  for (int rs = 0; rs < 2; ++rs)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 32 * wv + 16 * rs + 4 * lg + i;
      const WinRow x = win_row(r, tpr, G, w);
      ncs[rs][i] = -sC[r] * sl2;
      Z[rs][i] = 0.f;
      last[rs][i] = x.valid ? L - w + x.ii : -1;
    }
  // logits of key sub-tiles ks0 .. ks0 + 3 (16 keys each) of the tile in buffer buf
  auto mfma_half = [&](int buf, int ks0, f32x4 (&a)[2][4]) {
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&sK[buf][swzw(16 * (ks0 + ks) + l16, 4 * st + lg)]);
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        a[0][ks] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[0][st], kf, st == 0 ? z : a[0][ks], 0, 0, 0);
        a[1][ks] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[1][st], kf, st == 0 ? z : a[1][ks], 0, 0, 0);
      }
  };
  auto valu_half = [&](const f32x4 (&a)[2][4]) {
#pragma unroll
    for (int rs = 0; rs < 2; ++rs)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int i = 0; i < 4; ++i) Z[rs][i] += __builtin_amdgcn_exp2f(fmaf(a[rs][ks][i], sl2, ncs[rs][i]));
  };
  // one MFMA half interleaved with the exponentials of the other (step j reads fragment j + 2,
  // runs the two MFMAs of fragment j and two logits' exponentials; a scheduling barrier closes
  // the step); the order of the sums is that of valu_half
  auto interleaved = [&](int buf, int ks0, f32x4 (&a)[2][4], const f32x4 (&v)[2][4]) {
    auto frag = [&](int j) {
      return *reinterpret_cast<const bf16x8*>(&sK[buf][swzw(16 * (ks0 + (j & 3)) + l16, 4 * (j >> 2) + lg)]);
    };
    bf16x8 f[3];
    f[0] = frag(0);
    f[1] = frag(1);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (j + 2 < 16) f[(j + 2) % 3] = frag(j + 2);
      const int st = j >> 2, ks = j & 3;
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      a[0][ks] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[0][st], f[j % 3], st == 0 ? z : a[0][ks], 0, 0, 0);
      a[1][ks] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[1][st], f[j % 3], st == 0 ? z : a[1][ks], 0, 0, 0);
#pragma unroll
      for (int uu = 0; uu < 2; ++uu) {
        const int u = 2 * j + uu, rs = u >> 4, kv = (u >> 2) & 3, i = u & 3;
        Z[rs][i] += __builtin_amdgcn_exp2f(fmaf(v[rs][kv][i], sl2, ncs[rs][i]));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  f32x4 accA[2][4], accB[2][4];
  // bulk tiles: every key visible to every window row (keys below L - w + 1, the first row's
  // position, all inside the prompt); buffer parity counts from t0
  const int b_end = min(t1, (L - w + 1) / kSlice);
  // tile t0 in (this wave's part; then every wave's)
  if (t0 + 1 < t1) wait_vmcnt<NI>();
  else wait_vmcnt<0>();
  __syncthreads();
  if (t0 < b_end) mfma_half(0, 0, accA);
  for (int kt = t0; kt < b_end; ++kt) {
    const int b = (kt - t0) & 1;
    interleaved(b, 4, accB, accA);
    // tile kt + 1 (issued an iteration ago) in; after the barrier every wave is done with
    // buffer b, which takes tile kt + 2
    wait_vmcnt<0>();
    __syncthreads();
    if (kt + 2 < t1) issue(kt + 2, b);
    if (kt + 1 < b_end) interleaved(b ^ 1, 0, accA, accB);
    else valu_half(accB);
  }
  // edge tiles: keys past a row's position, and past the prompt, take no part
  for (int kt = max(t0, b_end); kt < t1; ++kt) {
    const int k0 = kt * kSlice, b = (kt - t0) & 1;
    mfma_half(b, 0, accA);
    mfma_half(b, 4, accB);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int rs = 0; rs < 2; ++rs)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float x = fmaf(hf == 0 ? accA[rs][ks][i] : accB[rs][ks][i], sl2, ncs[rs][i]);
            const int key = k0 + 16 * (4 * hf + ks) + l16;
            if (key > last[rs][i]) x = kMaskedW;
            Z[rs][i] += __builtin_amdgcn_exp2f(x);
          }
    wait_vmcnt<0>();
    __syncthreads();
    if (kt + 2 < t1) issue(kt + 2, b);
  }
  // ---- sums over the 16 lanes of each row group; the row's log2 normaliser (one part), or the
  // part's row sum and, from part 0, the reference (several parts: the columns kernel adds them)
#pragma unroll
  for (int rs = 0; rs < 2; ++rs)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float z = Z[rs][i];
      z = dpp_addw<0x128>(z);
      z = dpp_addw<0x124>(z);
      z = dpp_addw<0x122>(z);
      z = dpp_addw<0x121>(z);
      const int r = 32 * wv + 16 * rs + 4 * lg + i;
      if (l16 == 0) {
        const bool valid = last[rs][i] >= 0;
        if (valid && !(z < __builtin_inff())) {
          // a key far above the row's reference: the job is rescored exactly before selection
          atomicOr(P.counters, RKV_STATUS_REPAIRED);
          atomicOr(P.counters + (size_t)kCounterStride * (1 + job) + 1, 1u);
        }
        if (parts == 1) {
          // padding and overflowing rows: +inf, every probability 0
          P.lam[(size_t)job * R + r] = valid && z < __builtin_inff() ? sC[r] * sl2 + __builtin_log2f(z)
                                                                      : __builtin_inff();
        } else {
          P.stats[((size_t)job * parts + part) * R + r] = z;
          if (part == 0) P.ncl[(size_t)job * R + r] = valid ? sC[r] * sl2 : __builtin_inff();
        }
      }
    }
}

template <int NRT>
__global__ __launch_bounds__(256, 2) void window_cols_kernel(const PrefillLaunch P) {
  constexpr int R = NRT * 32, NT = 256, NCH = NRT / 2;   // NCH chunks of 64 rows (two row tiles)
  constexpr int PERQ = R * kHeadDim / 8 / NT;            // 16-byte query chunks per thread
  static_assert(NCH % 2 == 0, "chunks alternate between two accumulator sets");
  __shared__ __attribute__((aligned(16))) uint16_t sQ[R * kHeadDim];
  __shared__ __attribute__((aligned(16))) float sLam[R];
  __shared__ float sColH[2][kMaxRowTiles][kSlice];   // per query head: column sums of a block's keys
  const int tid = threadIdx.x, lane = tid & 63, lg = lane >> 4, l16 = lane & 15;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int L = P.seq_len, w = P.window, G = P.group, Hq = P.n_q_heads, Hkv = P.n_kv_heads, B = P.batch;
  const int nsl = P.n_slices, tpr = P.row_tiles_per_group * 32, NTH = P.row_tiles_per_group;
  const int nbg = (nsl + kColBlocks - 1) / kColBlocks;
  const int job = blockIdx.x / nbg, bg = blockIdx.x - job * nbg;
  const int h = job % Hkv, s = (job / Hkv) % B, slot = job / (Hkv * B);
  const PrefillLayer& ly = P.layer[slot];
  const bool snap = ly.rule == RKV_SNAPKV;
  const uint16_t* khead = ly.k + (size_t)(s * Hkv + h) * L * kHeadDim;
  const uint16_t* qjob = ly.q + (size_t)(s * Hq + h * G) * w * kHeadDim;
  const float sl2 = P.scale_log2, inv_g = 1.f / (float)G;
  const int npre = L - w, ph = P.pool_half;

  // ---- the job's query block (padding rows zero) and row normalisers into LDS
#pragma unroll
  for (int u = 0; u < PERQ; ++u) {
    const int c = tid + NT * u, row = c >> 4, ch = c & 15;
    const WinRow x = win_row(row, tpr, G, w);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (x.valid) v = *reinterpret_cast<const u32x4*>(qjob + (size_t)(x.g * w + x.ii) * kHeadDim + 8 * ch);
    *reinterpret_cast<u32x4*>(&sQ[swzw(row, ch)]) = v;
  }
  if (P.window_parts == 1) {
    for (int r = tid; r < R; r += NT) sLam[r] = P.lam[(size_t)job * R + r];
  } else {
    // the parts' row sums, added in part order; +inf for padding and overflowing rows
    const int parts = P.window_parts;
    for (int r = tid; r < R; r += NT) {
      const float c = P.ncl[(size_t)job * R + r];
      float z = 0.f;
      for (int q = 0; q < parts; ++q) z += P.stats[((size_t)job * parts + q) * R + r];
      sLam[r] = c < __builtin_inff() && z < __builtin_inff() ? c + __builtin_log2f(z) : __builtin_inff();
    }
  }
  // ---- this wave's 32 keys of block b as B-operand fragments (key 32 wv + 16 ks + l16)
  auto load_k = [&](int b, bf16x8 (&kf)[2][4]) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int key = min(b * kSlice + 32 * wv + 16 * ks + l16, L - 1);
#pragma unroll
      for (int st = 0; st < 4; ++st)
        kf[ks][st] = as_bf16x8w(*reinterpret_cast<const u32x4*>(khead + (size_t)key * kHeadDim + 8 * (4 * st + lg)));
    }
  };
  const int b0 = bg * kColBlocks, b1 = min(nsl, b0 + kColBlocks);
  bf16x8 kcur[2][4], knext[2][4];
  load_k(b0, kcur);
  __syncthreads();

  // Q fragment j = 4 st + rs of chunk c: rows 64 c + 16 rs + l16, 16-byte chunk 4 st + lg
  auto qfrag = [&](int c, int j) {
    return *reinterpret_cast<const bf16x8*>(&sQ[swzw(64 * c + 16 * (j & 3) + l16, 4 * (j >> 2) + lg)]);
  };
  // logits of chunk c: a[rs][ks][i] = row 64 c + 16 rs + 4 lg + i, key 32 wv + 16 ks + l16
  auto mfma_chunk = [&](int c, const bf16x8 (&kf)[2][4], f32x4 (&a)[4][2]) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int st = j >> 2, rs = j & 3;
      const bf16x8 qf = qfrag(c, j);
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      a[rs][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf, kf[0][st], st == 0 ? z : a[rs][0], 0, 0, 0);
      a[rs][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf, kf[1][st], st == 0 ? z : a[rs][1], 0, 0, 0);
    }
  };
  auto lam_chunk = [&](int c, f32x4 (&lm)[4]) {
#pragma unroll
    for (int rs = 0; rs < 4; ++rs) lm[rs] = *reinterpret_cast<const f32x4*>(&sLam[64 * c + 16 * rs + 4 * lg]);
  };
  // probabilities of a chunk's logits summed per lane into ct[row tile][ks]; value u of the 32 a
  // lane holds is (rs, ks, i) = (u / 8, (u / 4) % 2, u % 4)
  auto exps_plain = [&](const f32x4 (&a)[4][2], const f32x4 (&lm)[4], float (&ct)[2][2]) {
#pragma unroll
    for (int u = 0; u < 32; ++u) {
      const int rs = u >> 3, ks = (u >> 2) & 1, i = u & 3;
      ct[rs >> 1][ks] += __builtin_amdgcn_exp2f(fmaf(a[rs][ks][i], sl2, -lm[rs][i]));
    }
  };
  // blocks with keys past a row's position (or past the prompt): those keys and padding rows
  // take no part
  auto exps_masked = [&](int c, int kbase, const f32x4 (&a)[4][2], const f32x4 (&lm)[4], float (&ct)[2][2]) {
#pragma unroll
    for (int u = 0; u < 32; ++u) {
      const int rs = u >> 3, ks = (u >> 2) & 1, i = u & 3;
      float x = fmaf(a[rs][ks][i], sl2, -lm[rs][i]);
      const WinRow y = win_row(64 * c + 16 * rs + 4 * lg + i, tpr, G, w);
      if (!y.valid || kbase + 16 * ks + l16 > L - w + y.ii) x = kMaskedW;
      ct[rs >> 1][ks] += __builtin_amdgcn_exp2f(x);
    }
  };
  // the MFMAs of chunk cn against keys kf (into a) interleaved with the exponentials of the
  // previous chunk's logits v, in the order of exps_plain: step j reads Q fragment j + 2, runs
  // fragment j's two MFMAs and two exponentials; a scheduling barrier closes the step
  auto interleaved = [&](int cn, const bf16x8 (&kf)[2][4], f32x4 (&a)[4][2], const f32x4 (&v)[4][2],
                         const f32x4 (&lm)[4], float (&ct)[2][2]) {
    bf16x8 f[3];
    f[0] = qfrag(cn, 0);
    f[1] = qfrag(cn, 1);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (j + 2 < 16) f[(j + 2) % 3] = qfrag(cn, j + 2);
      const int st = j >> 2, rs = j & 3;
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      a[rs][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f[j % 3], kf[0][st], st == 0 ? z : a[rs][0], 0, 0, 0);
      a[rs][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f[j % 3], kf[1][st], st == 0 ? z : a[rs][1], 0, 0, 0);
#pragma unroll
      for (int uu = 0; uu < 2; ++uu) {
        const int u = 2 * j + uu, rv = u >> 3, ks = (u >> 2) & 1, i = u & 3;
        ct[rv >> 1][ks] += __builtin_amdgcn_exp2f(fmaf(v[rv][ks][i], sl2, -lm[rv][i]));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // sums over the wave's four row groups (lanes l, l ^ 32, then l ^ 16), then per query head:
  // row tile t = 2 c + tt belongs to head t / NTH; a head's sum runs over its tiles in order and
  // goes to sColH when its last tile is in (lanes 0-31: key 32 wv + 16 lg + l16)
  auto heads = [&](int c, int buf, float (&ct)[2][2], float (&hs)[2]) {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const auto p0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(ct[tt][ks]), __float_as_uint(ct[tt][ks]), false, false);
        const float v = __uint_as_float(p0[0]) + __uint_as_float(p0[1]);
        const auto p1 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        ct[tt][ks] = __uint_as_float(p1[0]) + __uint_as_float(p1[1]);
      }
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int t = 2 * c + tt;
      hs[0] += ct[tt][0];
      hs[1] += ct[tt][1];
      if ((t + 1) % NTH == 0) {
        const int g = t / NTH;
        if (g < G && lane < 32) sColH[buf][g][32 * wv + 16 * lg + l16] = lg == 0 ? hs[0] : hs[1];
        hs[0] = hs[1] = 0.f;
      }
    }
  };
  // scores of block b from the per-head column sums; thread = (key, query-head half)
  auto store = [&](int b, int buf) {
    const int cbase = b * kSlice, kl = tid >> 1, kk = cbase + kl;
    const int g0 = (tid & 1) * ((G + 1) >> 1), g1 = min(G, g0 + ((G + 1) >> 1));
    const float NEG_INF = -__builtin_inff();
    float su = 0.f, sc = 0.f;
    if (kk < L) {
      // max-pool window [lo, hi] inside the block and the prefix [0, L - w); clamping a
      // neighbour into it repeats a member, so the reads need no branches (for window keys the
      // pooled value is not used)
      const int lo = max(kk - ph, cbase) - cbase;
      const int hi = max(min(min(kk + ph, cbase + kSlice - 1), npre - 1) - cbase, lo);
      for (int g = g0; g < g1; ++g) {
        const float* cg = sColH[buf][g];
        su += cg[kl];
        if (snap) {
          float m = NEG_INF;
          if (ph == 3) {
            float x[7];
#pragma unroll
            for (int u = 0; u < 7; ++u) x[u] = cg[min(max(kl - 3 + u, lo), hi)];
#pragma unroll
            for (int u = 0; u < 7; ++u) m = fmaxf(m, x[u]);
          } else {
            for (int u = 0; u <= 2 * ph; ++u) m = fmaxf(m, cg[min(max(kl - ph + u, lo), hi)]);
          }
          sc += m;
        }
      }
    }
    su += __shfl_xor(su, 1);
    sc += __shfl_xor(sc, 1);
    if ((tid & 1) == 0 && kk < L) {
      su *= inv_g;
      P.S[(size_t)job * L + kk] = snap && kk < npre ? sc * inv_g : su;
      if (snap && P.want_unpooled) P.Su[(size_t)job * L + kk] = su;
    }
    if (snap && ph > 0) {   // slice-edge column sums per head: offsets [0, 2 ph) and [128 - 2 ph, 128)
      const int E = 4 * ph, twoP = 2 * ph;
      float* ed = P.edge + ((size_t)job * nsl + b) * G * E;
      for (int e2 = tid; e2 < G * E; e2 += NT) {
        const int g = e2 / E, o = e2 - g * E;
        const int kl2 = o < twoP ? o : kSlice - twoP + (o - twoP);
        ed[e2] = (cbase + kl2 < L) ? sColH[buf][g][kl2] : 0.f;
      }
    }
  };

  // The pipeline runs across blocks: the MFMAs of a block's first chunk go beside the previous
  // block's last exponentials when both blocks are free of masks for this wave (chained).
  int buf = 0;
  bool chained = false;   // accA holds chunk 0 of block b
  f32x4 accA[4][2], accB[4][2];
  for (int b = b0; b < b1; ++b, buf ^= 1) {
    if (b + 1 < b1) load_k(b + 1, knext);
    const int kbase = b * kSlice + 32 * wv;
    float hs[2] = {0.f, 0.f};
    f32x4 lm[4];
    if (kbase + 31 <= L - w) {
      // every key of the wave visible to every window row: chunk c + 1's MFMAs run beside chunk
      // c's exponentials
      const bool chain_next = b + 1 < b1 && kbase + kSlice + 31 <= L - w;
      if (!chained) mfma_chunk(0, kcur, accA);
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        float ct[2][2] = {{0.f, 0.f}, {0.f, 0.f}};
        lam_chunk(c, lm);
        if (c + 1 < NCH) {
          if ((c & 1) == 0) interleaved(c + 1, kcur, accB, accA, lm, ct);
          else interleaved(c + 1, kcur, accA, accB, lm, ct);
        } else if (chain_next) {
          interleaved(0, knext, accA, accB, lm, ct);   // NCH is even: the last chunk is in accB
        } else {
          exps_plain(accB, lm, ct);
        }
        heads(c, buf, ct, hs);
      }
      chained = chain_next;
    } else {
#pragma unroll 1
      for (int c = 0; c < NCH; ++c) {
        float ct[2][2] = {{0.f, 0.f}, {0.f, 0.f}};
        mfma_chunk(c, kcur, accA);
        lam_chunk(c, lm);
        exps_masked(c, kbase, accA, lm, ct);
        heads(c, buf, ct, hs);
      }
      chained = false;
    }
    __syncthreads();   // sColH[buf] complete; the buffer is written again two blocks later
    store(b, buf);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int st = 0; st < 4; ++st) kcur[ks][st] = knext[ks][st];
  }
}

template <int NRT>
int launch_window_nrt(const PrefillLaunch& P, int n_jobs, hipStream_t st) {
  window_rows_kernel<NRT><<<n_jobs * P.window_parts, NRT * 64, 0, st>>>(P);
  const int nbg = (P.n_slices + kColBlocks - 1) / kColBlocks;
  window_cols_kernel<NRT><<<(unsigned)((int64_t)n_jobs * nbg), 256, 0, st>>>(P);
  return (int)hipGetLastError();
}

}  // namespace

int launch_window(const PrefillLaunch& P, int row_tiles, void* stream) {
  const int n_jobs = P.batch * P.n_window * P.n_kv_heads;
  if (n_jobs <= 0) return 0;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return row_tiles <= 4 ? launch_window_nrt<4>(P, n_jobs, st) : launch_window_nrt<8>(P, n_jobs, st);
}

}  // namespace rkv
