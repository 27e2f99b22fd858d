// Attention-entropy layer score for capacity allocation (Section 3.3) on gfx950.
//
// H_l is the mean, over sequences, query heads and profiled query positions, of the Shannon
// entropy (nats) of each query's causal attention row: the softmax of q_t . k_j / sqrt(d) over
// keys j = 0..t, query head hq reading KV head hq / G.
//
// entropy_rows_kernel: one workgroup per (layer, sequence, KV head, block of 32 query
// positions), one wave per query head of the group.  The wave's query fragments stay in
// registers; the K tiles of 128 keys stream through two LDS buffers (prefetched into registers
// one tile ahead) and the logits z come from 16x16x32 bf16 MFMA, taken against a per-row
// reference c_t = max(logit with key t, logit with key 0) (both true logits of the row), so
// e = exp2(x) with x = (z - c) log2(e) / sqrt(d) stays finite unless a key beats the reference
// by more than ~88 natural-log units.  On tiles without masks the MFMAs of one half-tile run
// interleaved with the exponentials of the other half.  Per row the lane keeps Z = sum e and T = sum e x over its
// keys; the 16 lanes of a row meet once at the end, and
//   H = -sum p ln p = ln 2 (log2 Z - T / Z).
// A non-finite row is written as it is and reported by the averaging kernel.
// Each workgroup also leaves the double-precision sum of its rows; entropy_mean_kernel (one
// workgroup per layer) adds those in a fixed order.
#include <hip/hip_runtime.h>

#include <math.h>

#include "rkv_internal.h"

namespace rkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kEntRows = 32;    // query positions per workgroup (two 16-row MFMA sub-tiles)
constexpr float kMasked = -1e30f;   // exponent of a key a row does not see: exp2 gives 0, 0 * x = 0

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int CTRL>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}

template <int G>
__global__ __launch_bounds__(64 * (G > 4 ? G : 4), 2) void entropy_rows_kernel(const EntropyLaunch E) {
  constexpr int NW = G > 4 ? G : 4;   // at least four waves share the K tile loads
  constexpr int NT = 64 * NW;
  constexpr int PER = kSlice * kHeadDim / 8 / NT;   // 16-byte K chunks per thread per tile
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kSlice * kHeadDim];   // double-buffered K tile
  __shared__ float sC[NW][kEntRows];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, lg = lane >> 4, l16 = lane & 15;
  const int L = E.seq_len, n_q = E.n_q, Hq = E.n_q_heads, Hkv = E.n_kv_heads;
  const int nqb = (n_q + kEntRows - 1) / kEntRows;
  int item = blockIdx.x;
  const int qb = item % nqb;
  item /= nqb;
  const int h = item % Hkv;
  item /= Hkv;
  const int b = item % E.batch;
  const int layer = item / E.batch;
  const bool compute = wv < G;          // wave-uniform: one wave per query head of the group
  const int hq = h * G + (compute ? wv : 0);
  const int i0 = qb * kEntRows;            // first profiled query index of the block
  const int t0 = L - n_q + i0;             // its position
  const uint16_t* qrows = E.q[layer] + (size_t)(b * Hq + hq) * n_q * kHeadDim;
  const uint16_t* khead = E.k[layer] + (size_t)(b * Hkv + h) * L * kHeadDim;
  if (blockIdx.x == 0 && tid == 0 && E.first_group) E.status[0] = 0u;   // once per call: later launches OR into it

  // ---- per-row reference: lanes 0..31 of each wave take one row each
  if (compute && lane < kEntRows) {
    const int i = i0 + lane;
    float zd = 0.f, zs = 0.f;
    if (i < n_q) {
      const int t = L - n_q + i;
      const u32x4* qp = reinterpret_cast<const u32x4*>(qrows + (size_t)i * kHeadDim);
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
  // ---- query fragments (A operand): row 16 rs + l16, k-chunk 4 st + lg
  bf16x8 qa[2][4];
#pragma unroll
  for (int rs = 0; rs < 2; ++rs) {
    const int i = i0 + 16 * rs + l16;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (i < n_q) v = *reinterpret_cast<const u32x4*>(qrows + (size_t)i * kHeadDim + 8 * (4 * st + lg));
      qa[rs][st] = as_bf16x8(v);
    }
  }
  // ---- K tiles: keys [0, t_last] where t_last is the block's last valid position.  Tiles
  // whose keys every row of the block sees (k0 + 127 <= t0) are "bulk" tiles; the rest (at most
  // two) need the causal mask.
  const int t_last = L - n_q + min(i0 + kEntRows, n_q) - 1;
  const int n_tiles = t_last / kSlice + 1;
  const int n_bulk = min((t0 + 1) / kSlice, n_tiles);
  u32x4 pre[PER];
  auto fetch = [&](int kt) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int c = tid + NT * u, key = c >> 4, ch = c & 15;
      const int kk = min(kt * kSlice + key, L - 1);   // keys past the prompt are masked below
      pre[u] = *reinterpret_cast<const u32x4*>(khead + (size_t)kk * kHeadDim + 8 * ch);
    }
  };
  auto put = [&](int buf) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int c = tid + NT * u, key = c >> 4, ch = c & 15;
      *reinterpret_cast<u32x4*>(&sK[buf][(key * 16 + (ch ^ (key & 15))) * 8]) = pre[u];
    }
  };
  fetch(0);
  __syncthreads();   // sC written
  const float sl2 = E.scale_log2;
  float ncs[2][4];   // -c sl2 per row
#pragma unroll
  for (int rs = 0; rs < 2; ++rs)
#pragma unroll
    for (int i = 0; i < 4; ++i) ncs[rs][i] = -sC[wv][16 * rs + 4 * lg + i] * sl2;
  float Z[2][4], T[2][4];
#pragma unroll
  for (int rs = 0; rs < 2; ++rs)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      Z[rs][i] = 0.f;
      T[rs][i] = 0.f;
    }
  // logits of key sub-tiles ks0 .. ks0 + 3 of the tile in buffer buf (x = q.k, the reference is
  // applied with the scale afterwards)
  auto mfma_half = [&](int buf, int ks0, f32x4 (&a)[2][4]) {
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int key = 16 * (ks0 + ks) + l16, ch = 4 * st + lg;
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&sK[buf][(key * 16 + (ch ^ (key & 15))) * 8]);
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        a[0][ks] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[0][st], kf, st == 0 ? z : a[0][ks], 0, 0, 0);
        a[1][ks] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[1][st], kf, st == 0 ? z : a[1][ks], 0, 0, 0);
      }
  };
  // exponentials and the row sums Z (of e) and T (of e x) for four key sub-tiles
  auto valu_half = [&](const f32x4 (&a)[2][4]) {
#pragma unroll
    for (int rs = 0; rs < 2; ++rs)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float x = fmaf(a[rs][ks][i], sl2, ncs[rs][i]);
          const float e = __builtin_amdgcn_exp2f(x);
          Z[rs][i] += e;
          T[rs][i] = fmaf(e, x, T[rs][i]);
        }
  };
  // one MFMA half (into a) interleaved with the exponentials of the other half (from v): step j
  // reads K fragment j + 2, runs the two MFMAs of fragment j and the exponentials of two
  // logits; a scheduling barrier closes each step, so every fragment is read two steps before
  // its MFMAs.  Fragment j is (st, ks) = (j / 4, j % 4); logit u of v is (rs, ks, i) =
  // (u / 16, (u / 4) % 4, u % 4).  The sums keep the order of valu_half.
  auto interleaved = [&](int buf, int ks0, f32x4 (&a)[2][4], const f32x4 (&v)[2][4]) {
    auto frag = [&](int j) {
      const int key = 16 * (ks0 + (j & 3)) + l16, ch = 4 * (j >> 2) + lg;
      return *reinterpret_cast<const bf16x8*>(&sK[buf][(key * 16 + (ch ^ (key & 15))) * 8]);
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
        const float x = fmaf(v[rs][kv][i], sl2, ncs[rs][i]);
        const float e = __builtin_amdgcn_exp2f(x);
        Z[rs][i] += e;
        T[rs][i] = fmaf(e, x, T[rs][i]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  f32x4 accA[2][4], accB[2][4];
  // bulk tiles, software-pipelined: MFMA half B of tile kt with the exponentials of half A, then
  // (after the barrier that publishes tile kt + 1) MFMA half A of tile kt + 1 with the
  // exponentials of half B of tile kt.  The order of the sums is that of the plain loop.
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
  // edge tiles: keys past a row's position (and past the prompt) take no part
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
              const int key = k0 + 16 * (4 * hf + ks) + l16;
              const int ir = i0 + 16 * rs + 4 * lg + i;
              if (key > L - n_q + ir || ir >= n_q) x = kMasked;
              const float e = __builtin_amdgcn_exp2f(x);
              Z[rs][i] += e;
              T[rs][i] = fmaf(e, x, T[rs][i]);
            }
    }
    if (kt + 1 < n_tiles) {
      put((kt + 1) & 1);
      if (kt + 2 < n_tiles) fetch(kt + 2);
    }
    __syncthreads();
  }
  // ---- the 16 lanes of each row (one DPP row) add up; lane l16 == 0 writes the entropy and
  // adds it to the workgroup's partial sum (fixed order: lanes, then waves)
  double part = 0.0;
#pragma unroll
  for (int rs = 0; rs < 2; ++rs)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float z = Z[rs][i], tt = T[rs][i];
      z = dpp_add<0x128>(z);   // row_ror:8
      z = dpp_add<0x124>(z);   // row_ror:4
      z = dpp_add<0x122>(z);   // row_ror:2
      z = dpp_add<0x121>(z);   // row_ror:1
      tt = dpp_add<0x128>(tt);
      tt = dpp_add<0x124>(tt);
      tt = dpp_add<0x122>(tt);
      tt = dpp_add<0x121>(tt);
      const int ir = i0 + 16 * rs + 4 * lg + i;
      if (compute && l16 == 0 && ir < n_q) {
        const float H = 0.6931471805599453f * (__builtin_log2f(z) - tt / z);
        E.rows[((size_t)(layer * E.batch + b) * Hq + hq) * n_q + ir] = H;
        part += (double)H;
      }
    }
  __shared__ double sPart[NW];
#pragma unroll
  for (int o = 16; o < 64; o <<= 1) part += __shfl_xor(part, o);   // lanes 0, 16, 32, 48
  if (lane == 0) sPart[wv] = part;
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
    for (int w = 0; w < G; ++w) t += sPart[w];
    E.partial[blockIdx.x] = t;   // blocks of one layer are consecutive
  }
}

__global__ __launch_bounds__(256) void entropy_mean_kernel(const EntropyLaunch E) {
  __shared__ double sSum[256];
  __shared__ int sBad;
  const int tid = threadIdx.x, layer = blockIdx.x;
  const size_t n = (size_t)E.batch * E.n_q_heads * E.n_q;
  const int nb = E.batch * E.n_kv_heads * ((E.n_q + kEntRows - 1) / kEntRows);   // row blocks per layer
  const double* part = E.partial + (size_t)layer * nb;
  if (tid == 0) sBad = 0;
  __syncthreads();
  double s = 0.0;
  for (int r = tid; r < nb; r += 256) s += part[r];
  // a non-finite row makes its block's partial sum non-finite
  if (!(fabs(s) < __builtin_inf())) sBad = 1;
  sSum[tid] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (tid < o) sSum[tid] += sSum[tid + o];
    __syncthreads();
  }
  if (tid == 0) {
    E.h[layer] = (float)(sSum[0] / (double)n);
    if (sBad) atomicOr(E.status, 1u);
  }
}

}  // namespace

int launch_entropy(const EntropyLaunch& E, void* stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int G = E.n_q_heads / E.n_kv_heads;
  const unsigned grid = (unsigned)(E.n_layers * E.batch * E.n_kv_heads * ((E.n_q + kEntRows - 1) / kEntRows));
  switch (G) {
    case 1: entropy_rows_kernel<1><<<grid, 256, 0, st>>>(E); break;
    case 2: entropy_rows_kernel<2><<<grid, 256, 0, st>>>(E); break;
    case 4: entropy_rows_kernel<4><<<grid, 256, 0, st>>>(E); break;
    case 8: entropy_rows_kernel<8><<<grid, 512, 0, st>>>(E); break;
    default: return (int)hipErrorInvalidValue;
  }
  entropy_mean_kernel<<<E.n_layers, 256, 0, st>>>(E);
  return (int)hipGetLastError();
}

}  // namespace rkv
