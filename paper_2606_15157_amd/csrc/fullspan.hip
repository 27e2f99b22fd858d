// H2O prefill with full-span accumulation on gfx950: the score of key j is the group mean of the
// attention it receives from every prompt query t >= j (H2O's accumulated attention, Section 2.1),
//   S[h, j] = (1/G) sum_g sum_{t >= j} softmax_j(q[hG+g, t] . k[h, .] / sqrt(d)) over keys <= t.
// Two passes over the causal logits, no atomics, fixed summation order:
//
// fullspan_rows_kernel: one workgroup per (job, 32 query positions), one wave per query head of
//   the group.  The wave's query fragments stay in registers, 128-key tiles stream through two
//   LDS buffers, bf16 MFMA logits are taken against a fixed per-row reference c_t = max(logit with key t,
//   logit with key 0); the row's log2 normaliser Lambda_t = c_t log2(e)/sqrt(d) + log2(sum_j
//   exp2(x_tj - c_t log2(e)/sqrt(d))) goes to the workspace.  A non-finite normaliser (a key
//   beyond ~88 natural-log units above the reference) sets status bit 1.
// fullspan_cols_kernel: one workgroup per (job, 128-key block), four waves of 32 keys each; the
//   wave's key fragments stay in registers, 128-row query tiles (G heads x 128/G positions) at or
//   after the block stream through LDS with their normalisers, and each lane sums
//   p = exp2(x - Lambda_t) over its rows; the four lane groups meet once at the end.
// In both, tiles without masks run software-pipelined: the MFMAs of one half-tile interleave
// with the exponentials of the other half, in the summation order of the plain loop.
// Jobs here are the full-span ones: job = (slot * B + b) * Hkv + h with slot >= n_window.
#include <hip/hip_runtime.h>

#include <math.h>

#include "rkv_internal.h"

namespace rkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kFsRows = 32;          // query positions per row-pass workgroup
constexpr float kMasked = -1e30f;    // exponent of a hidden key: exp2 gives 0

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int CTRL>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}

// LDS position of 16-byte chunk `ch` of row `row` of a 128 x 128 bf16 tile (XOR swizzle: the
// 16 rows a fragment read touches hit distinct banks)
__device__ __forceinline__ int swz(int row, int ch) { return (row * 16 + (ch ^ (row & 15))) * 8; }

template <int G>
__global__ __launch_bounds__(64 * (G > 4 ? G : 4), 2) void fullspan_rows_kernel(const PrefillLaunch P) {
  constexpr int NW = G > 4 ? G : 4;
  constexpr int NT = 64 * NW;
  constexpr int PER = kSlice * kHeadDim / 8 / NT;
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kSlice * kHeadDim];   // double-buffered K tile
  __shared__ float sC[NW][kFsRows];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, lg = lane >> 4, l16 = lane & 15;
  const int L = P.seq_len, Hq = P.n_q_heads, Hkv = P.n_kv_heads, B = P.batch;
  const int nqb = (L + kFsRows - 1) / kFsRows;
  const int jf = blockIdx.x / nqb, qb = blockIdx.x - jf * nqb;
  const int job = B * Hkv * P.n_window + jf;
  const int h = job % Hkv, s = (job / Hkv) % B, slot = job / (Hkv * B);
  const PrefillLayer& ly = P.layer[slot];
  const bool compute = wv < G;
  const int g = compute ? wv : 0, hq = h * G + g;
  const int t0 = qb * kFsRows;
  const uint16_t* qrows = ly.q + (size_t)(s * Hq + hq) * L * kHeadDim;
  const uint16_t* khead = ly.k + (size_t)(s * Hkv + h) * L * kHeadDim;
  float* lam = P.lamf + ((size_t)jf * G + g) * L;

  if (compute && lane < kFsRows) {
    const int t = t0 + lane;
    float zd = 0.f, zs = 0.f;
    if (t < L) {
      const u32x4* qp = reinterpret_cast<const u32x4*>(qrows + (size_t)t * kHeadDim);
      const u32x4* kd = reinterpret_cast<const u32x4*>(khead + (size_t)t * kHeadDim);
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
    sC[wv][lane] = fmaxf(zd, zs);
  }
  bf16x8 qa[2][4];
#pragma unroll
  for (int rs = 0; rs < 2; ++rs) {
    const int t = t0 + 16 * rs + l16;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (t < L) v = *reinterpret_cast<const u32x4*>(qrows + (size_t)t * kHeadDim + 8 * (4 * st + lg));
      qa[rs][st] = as_bf16x8(v);
    }
  }
  const int t_last = min(t0 + kFsRows, L) - 1;
  const int n_tiles = t_last / kSlice + 1;
  const int n_bulk = min((t0 + 1) / kSlice, n_tiles);   // tiles every row of the block sees whole
  u32x4 pre[PER];
  auto fetch = [&](int kt) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int c = tid + NT * u, key = c >> 4, ch = c & 15;
      const int kk = min(kt * kSlice + key, L - 1);
      pre[u] = *reinterpret_cast<const u32x4*>(khead + (size_t)kk * kHeadDim + 8 * ch);
    }
  };
  auto put = [&](int buf) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int c = tid + NT * u, key = c >> 4, ch = c & 15;
      *reinterpret_cast<u32x4*>(&sK[buf][swz(key, ch)]) = pre[u];
    }
  };
  fetch(0);
  __syncthreads();
  const float sl2 = P.scale_log2;
  float cref[2][4], ncs[2][4], Z[2][4];
#pragma unroll
  for (int rs = 0; rs < 2; ++rs)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      cref[rs][i] = sC[wv][16 * rs + 4 * lg + i];
      ncs[rs][i] = -cref[rs][i] * sl2;
      Z[rs][i] = 0.f;
    }
  // logits (q.k) of key sub-tiles ks0 .. ks0 + 3 of the tile in buffer buf
  auto mfma_half = [&](int buf, int ks0, f32x4 (&a)[2][4]) {
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&sK[buf][swz(16 * (ks0 + ks) + l16, 4 * st + lg)]);
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
  // one MFMA half (into a) interleaved with the exponentials of the other half (from v): step j
  // reads K fragment j + 2, runs the two MFMAs of fragment j and the exponentials of two
  // logits, and a scheduling barrier closes the step.  Fragment j is (st, ks) = (j / 4, j % 4);
  // logit u of v is (rs, ks, i) = (u / 16, (u / 4) % 4, u % 4), the order of valu_half.
  auto interleaved = [&](int buf, int ks0, f32x4 (&a)[2][4], const f32x4 (&v)[2][4]) {
    auto frag = [&](int j) {
      return *reinterpret_cast<const bf16x8*>(&sK[buf][swz(16 * (ks0 + (j & 3)) + l16, 4 * (j >> 2) + lg)]);
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
  // bulk tiles, software-pipelined: MFMA half B of tile kt with the exponentials of half A, then
  // (after the barrier that publishes tile kt + 1) MFMA half A of tile kt + 1 with the
  // exponentials of half B of tile kt; the sums keep the order of the plain loop
  put(0);
  if (n_tiles > 1) fetch(1);
  __syncthreads();
  if (compute && n_bulk > 0) mfma_half(0, 0, accA);
  for (int kt = 0; kt < n_bulk; ++kt) {
    if (compute) interleaved(kt & 1, 4, accB, accA);
    if (kt + 1 < n_tiles) {
      put((kt + 1) & 1);
      if (kt + 2 < n_tiles) fetch(kt + 2);
    }
    __syncthreads();   // tile kt + 1 published; every wave is done with tile kt's buffer
    if (compute) {
      if (kt + 1 < n_bulk) {
        interleaved((kt + 1) & 1, 0, accA, accB);
      } else {
        valu_half(accB);
      }
    }
  }
  // edge tiles: keys past a row's position (and rows past the prompt) take no part
  for (int kt = n_bulk; kt < n_tiles; ++kt) {
    if (compute) {
      const int k0 = kt * kSlice;
      mfma_half(kt & 1, 0, accA);
      mfma_half(kt & 1, 4, accB);
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int rs = 0; rs < 2; ++rs)
#pragma unroll
          for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float av = hf == 0 ? accA[rs][ks][i] : accB[rs][ks][i];
              float x = fmaf(av, sl2, ncs[rs][i]);
              const int key = k0 + 16 * (4 * hf + ks) + l16, t = t0 + 16 * rs + 4 * lg + i;
              if (key > t || t >= L) x = kMasked;
              Z[rs][i] += __builtin_amdgcn_exp2f(x);
            }
    }
    if (kt + 1 < n_tiles) {
      put((kt + 1) & 1);
      if (kt + 2 < n_tiles) fetch(kt + 2);
    }
    __syncthreads();
  }
  if (!compute) return;
#pragma unroll
  for (int rs = 0; rs < 2; ++rs)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float z = Z[rs][i];
      z = dpp_add<0x128>(z);
      z = dpp_add<0x124>(z);
      z = dpp_add<0x122>(z);
      z = dpp_add<0x121>(z);
      const int t = t0 + 16 * rs + 4 * lg + i;
      if (l16 == 0 && t < L) {
        const float lm = cref[rs][i] * sl2 + __builtin_log2f(z);
        if (!(z < __builtin_inff())) atomicOr(P.counters, 2u);
        lam[t] = lm;
      }
    }
}

template <int G>
__global__ __launch_bounds__(256, 2) void fullspan_cols_kernel(const PrefillLaunch P) {
  constexpr int NT = 256;
  constexpr int PT = 128 / G;                      // query positions per 128-row tile
  constexpr int PER = 128 * kHeadDim / 8 / NT;     // 16-byte chunks of the query tile per thread
  __shared__ __attribute__((aligned(16))) uint16_t sQ[2][128 * kHeadDim];   // double-buffered tiles
  // the row normalisers of tile it sit in sLam[it % 3]: the exponentials of a tile's second half
  // run after the barrier that publishes the next tile, while faster waves may already write the
  // tile after that
  __shared__ float sLam[3][128];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, lg = lane >> 4, l16 = lane & 15;
  const int L = P.seq_len, Hq = P.n_q_heads, Hkv = P.n_kv_heads, B = P.batch;
  const int nkb = (L + kSlice - 1) / kSlice;
  const int jf = blockIdx.x / nkb, kb = blockIdx.x - jf * nkb;
  const int job = B * Hkv * P.n_window + jf;
  const int h = job % Hkv, s = (job / Hkv) % B, slot = job / (Hkv * B);
  const PrefillLayer& ly = P.layer[slot];
  const int j0 = kb * kSlice;
  const uint16_t* khead = ly.k + (size_t)(s * Hkv + h) * L * kHeadDim;
  const uint16_t* qbase = ly.q + (size_t)(s * Hq + h * G) * L * kHeadDim;   // the group's first head
  const float* lamj = P.lamf + (size_t)jf * G * L;

  // this wave's 32 keys as B-operand fragments: key j0 + 32 wv + 16 ks + l16, chunk 4 st + lg
  bf16x8 kf[2][4];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int key = min(j0 + 32 * wv + 16 * ks + l16, L - 1);   // keys past the prompt are unused
#pragma unroll
    for (int st = 0; st < 4; ++st)
      kf[ks][st] = as_bf16x8(*reinterpret_cast<const u32x4*>(khead + (size_t)key * kHeadDim + 8 * (4 * st + lg)));
  }
  // query tiles: positions [t0, t0 + PT) of every head of the group, from the tile holding j0
  const int tfirst = (j0 / PT) * PT;
  const int n_tiles = (L - tfirst + PT - 1) / PT;
  u32x4 pre[PER];
  float lpre = 0.f;
  auto fetch = [&](int it) {
    const int t0 = tfirst + it * PT;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int c = tid + NT * u, row = c >> 4, ch = c & 15;
      const int gg = row / PT, t = min(t0 + (row - gg * PT), L - 1);
      pre[u] = *reinterpret_cast<const u32x4*>(qbase + ((size_t)gg * L + t) * kHeadDim + 8 * ch);
    }
    if (tid < 128) {
      const int gg = tid / PT, t = t0 + (tid - gg * PT);
      lpre = t < L ? lamj[(size_t)gg * L + t] : 0.f;
    }
  };
  auto put = [&](int it) {   // tile it (in registers) into sQ[it % 2], sLam[it % 3]
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int c = tid + NT * u, row = c >> 4, ch = c & 15;
      *reinterpret_cast<u32x4*>(&sQ[it & 1][swz(row, ch)]) = pre[u];
    }
    if (tid < 128) sLam[it % 3][tid] = lpre;
  };
  const float sl2 = P.scale_log2;
  float col[2] = {0.f, 0.f};
  // logits of row sub-tiles rs0 .. rs0 + 3 of the tile in buffer buf against this wave's keys
  auto mfma_half = [&](int buf, int rs0, f32x4 (&a)[4][2]) {
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int rs = 0; rs < 4; ++rs) {
        const bf16x8 qa = *reinterpret_cast<const bf16x8*>(&sQ[buf][swz(16 * (rs0 + rs) + l16, 4 * st + lg)]);
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        a[rs][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa, kf[0][st], st == 0 ? z : a[rs][0], 0, 0, 0);
        a[rs][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa, kf[1][st], st == 0 ? z : a[rs][1], 0, 0, 0);
      }
  };
  // probabilities of those rows summed per key (no mask: a bulk tile)
  auto valu_half = [&](int it, int rs0, const f32x4 (&a)[4][2]) {
#pragma unroll
    for (int rs = 0; rs < 4; ++rs) {
      const f32x4 lm = *reinterpret_cast<const f32x4*>(&sLam[it % 3][16 * (rs0 + rs) + 4 * lg]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) col[ks] += __builtin_amdgcn_exp2f(fmaf(a[rs][ks][i], sl2, -lm[i]));
    }
  };
  // one MFMA half (row sub-tiles rs0 .. rs0 + 3 of tile `buf` into a) interleaved with the
  // probabilities of the other half (rows vr0 .. vr0 + 3 of tile vit, from v): step j reads query
  // fragment j + 2, runs the two MFMAs of fragment j and two logits' exponentials, and a
  // scheduling barrier closes the step.  Fragment j is (st, rs) = (j / 4, j % 4); logit u of v is
  // (rs, i, ks) = (u / 8, (u / 2) % 4, u % 2), the order of valu_half.
  auto interleaved = [&](int buf, int rs0, f32x4 (&a)[4][2], int vit, int vr0, const f32x4 (&v)[4][2]) {
    auto frag = [&](int j) {
      return *reinterpret_cast<const bf16x8*>(&sQ[buf][swz(16 * (rs0 + (j & 3)) + l16, 4 * (j >> 2) + lg)]);
    };
    // the normalisers of the exponential half first (LDS reads complete in order)
    f32x4 lm4[4];
#pragma unroll
    for (int vr = 0; vr < 4; ++vr) lm4[vr] = *reinterpret_cast<const f32x4*>(&sLam[vit % 3][16 * (vr0 + vr) + 4 * lg]);
    bf16x8 f[3];
    f[0] = frag(0);
    f[1] = frag(1);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (j + 2 < 16) f[(j + 2) % 3] = frag(j + 2);
      const int st = j >> 2, rs = j & 3;
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      a[rs][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f[j % 3], kf[0][st], st == 0 ? z : a[rs][0], 0, 0, 0);
      a[rs][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f[j % 3], kf[1][st], st == 0 ? z : a[rs][1], 0, 0, 0);
#pragma unroll
      for (int uu = 0; uu < 2; ++uu) {
        const int u = 2 * j + uu, vr = u >> 3, i = (u >> 1) & 3, ks = u & 1;
        col[ks] += __builtin_amdgcn_exp2f(fmaf(v[vr][ks][i], sl2, -lm4[vr][i]));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  f32x4 accA[4][2], accB[4][2];
  // a tile with masks (near the diagonal, or past the prompt): rows 16 rs + 4 lg + i are head
  // (row / PT) at position t0 + row % PT; hidden keys and rows past the prompt contribute 0
  auto edge_tile = [&](int it) {
    const int t0 = tfirst + it * PT;
    mfma_half(it & 1, 0, accA);
    mfma_half(it & 1, 4, accB);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int rs = 0; rs < 4; ++rs) {
        const f32x4 lm = *reinterpret_cast<const f32x4*>(&sLam[it % 3][16 * (4 * hf + rs) + 4 * lg]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            float x = fmaf(hf == 0 ? accA[rs][ks][i] : accB[rs][ks][i], sl2, -lm[i]);
            const int row = 16 * (4 * hf + rs) + 4 * lg + i, t = t0 + row % PT;
            const int key = j0 + 32 * wv + 16 * ks + l16;
            if (key > t || t >= L) x = kMasked;
            col[ks] += __builtin_amdgcn_exp2f(x);
          }
      }
  };
  // publish tile it + 1 (already in registers) and request tile it + 2
  auto advance = [&](int it) {
    if (it + 1 < n_tiles) {
      put(it + 1);
      if (it + 2 < n_tiles) fetch(it + 2);
    }
    __syncthreads();
  };
  fetch(0);
  put(0);
  if (n_tiles > 1) fetch(1);
  __syncthreads();
  // tiles [it_lo, it_end) need no mask (every key at or before every row, every row inside the
  // prompt); they run software-pipelined as in the row pass, the others plainly, in tile order
  const int it_end = min(n_tiles, (L - tfirst) / PT);
  const int it_lo = min(it_end, (j0 + kSlice - 1 - tfirst + PT - 1) / PT);
  int it = 0;
  for (; it < it_lo; ++it) {
    edge_tile(it);
    advance(it);
  }
  if (it < it_end) {
    mfma_half(it & 1, 0, accA);
    for (; it < it_end; ++it) {
      interleaved(it & 1, 4, accB, it, 0, accA);
      advance(it);
      if (it + 1 < it_end) {
        interleaved((it + 1) & 1, 0, accA, it, 4, accB);
      } else {
        valu_half(it, 4, accB);
      }
    }
  }
  for (; it < n_tiles; ++it) {
    edge_tile(it);
    advance(it);
  }
  // sum over the four lane groups (rows 4 lg + i): lanes l, l ^ 32, then l ^ 16
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const auto p0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(col[ks]), __float_as_uint(col[ks]), false, false);
    float c = __uint_as_float(p0[0]) + __uint_as_float(p0[1]);
    const auto p1 = __builtin_amdgcn_permlane16_swap(__float_as_uint(c), __float_as_uint(c), false, false);
    c = __uint_as_float(p1[0]) + __uint_as_float(p1[1]);
    col[ks] = c;
  }
  // lane group ks writes key sub-tile ks
  if (lg < 2) {
    const int j = j0 + 32 * wv + 16 * lg + l16;
    if (j < L) P.S[(size_t)job * L + j] = (lg == 0 ? col[0] : col[1]) * (1.f / (float)G);
  }
}

}  // namespace

int launch_fullspan(const PrefillLaunch& P, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int n_full = P.batch * P.n_full * P.n_kv_heads;
  if (n_full <= 0) return 0;
  const int L = P.seq_len, G = P.group;
  const unsigned g_rows = (unsigned)(n_full * ((L + kFsRows - 1) / kFsRows));
  const unsigned g_cols = (unsigned)(n_full * ((L + kSlice - 1) / kSlice));
  switch (G) {
    case 1:
      fullspan_rows_kernel<1><<<g_rows, 256, 0, st>>>(P);
      fullspan_cols_kernel<1><<<g_cols, 256, 0, st>>>(P);
      break;
    case 2:
      fullspan_rows_kernel<2><<<g_rows, 256, 0, st>>>(P);
      fullspan_cols_kernel<2><<<g_cols, 256, 0, st>>>(P);
      break;
    case 4:
      fullspan_rows_kernel<4><<<g_rows, 256, 0, st>>>(P);
      fullspan_cols_kernel<4><<<g_cols, 256, 0, st>>>(P);
      break;
    case 8:
      fullspan_rows_kernel<8><<<g_rows, 512, 0, st>>>(P);
      fullspan_cols_kernel<8><<<g_cols, 256, 0, st>>>(P);
      break;
    default:
      return (int)hipErrorInvalidValue;
  }
  return (int)hipGetLastError();
}

}  // namespace rkv
