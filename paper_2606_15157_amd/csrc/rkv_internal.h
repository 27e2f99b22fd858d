// Internal declarations shared by the host code and the HIP kernels of librkv.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/rkv.h"

namespace rkv {

constexpr int kHeadDim = 128;      // head_dim the kernels are built for
constexpr int kMaxLayersPerLaunch = 32;
constexpr int kChunk = 768;        // keys per scoring work item (4 waves x 6 tiles of 32)
constexpr int kMaxRowTiles = 8;    // G * ceil(w / 32) supported by the scoring kernel
constexpr int kMaxPoolHalf = 64;   // pool_kernel / 2 supported
constexpr int kGatherParts = 4;    // gather work items per (sequence, layer, KV head)

// Per-layer work description of one prefill launch group.
struct PrefillLayer {
  const uint16_t* q;      // [B, Hq, w, d]
  const uint16_t* k;      // [B, Hkv, L, d]
  const uint16_t* v;      // [B, Hkv, L, d]
  uint16_t* k_out;        // [B, Hkv, n_keep, d]
  uint16_t* v_out;
  int32_t* idx;           // [B, Hkv, n_keep]
  float* score;           // [B, Hkv, L] or null
  float* acc;             // [B, Hkv, n_keep] or null
  int32_t rule;           // rkv_rule
  int32_t n_keep;         // retained rows per (sequence, KV head)
  int32_t cand_end;       // candidates [0, cand_end) (scored rules) / sink count (streaming)
  int32_t k_sel;          // number of candidates selected
  int32_t forced_lo;      // always-kept tail [forced_lo, forced_hi)
  int32_t forced_hi;
  int32_t slot;           // scored-layer slot (index into workspace regions), -1 if unscored
  int32_t all;            // 1: every position kept (FULL or b >= L)
};

// One launch of the fused eviction kernel over a group of up to 32 layers.
// Work items, in ticket order (ticket = atomic counter, so items start in this order):
//   step s: stats items of head s, score items of head s - lag_score, the select item of head
//   s - lag_score - lag_select and the gather items of head s - lag_score - lag_select -
//   lag_gather; then the copy items of the layers that are not scored.  Heads are (scored slot, sequence, KV head) triples.
struct PrefillLaunch {
  PrefillLayer layer[kMaxLayersPerLaunch];
  int32_t n_layers;
  int32_t n_scored;
  int32_t batch, seq_len, n_q_heads, n_kv_heads, window;
  int32_t group;          // G = Hq / Hkv
  int32_t row_tiles_per_group;  // ceil(w / 32)
  int32_t n_chunks;       // ceil(L / kChunk)
  int32_t pool_half;      // pool_kernel / 2
  int32_t want_unpooled;  // write the unpooled score array (acc seeding) for SnapKV layers
  int32_t lag_score;      // steps from a head's stats items to its score items
  int32_t lag_select;     // steps from its score items to its select item
  int32_t lag_gather;     // steps from its select item to its gather items
  int32_t n_unscored;     // layers copied without scoring
  int32_t n_tickets;      // total work items (= grid size)
  float scale_log2;       // log2(e) / sqrt(d)
  // workspace regions
  uint32_t* counters;     // [0] status, [1] unused, then per head: selection done
  // stats .. edge are contiguous; the reset kernel fills them with NaN ("not written yet")
  float* stats;           // [n_heads][n_chunks][R][2]  chunk row max (log2 units) / sum
  int64_t fill_vec4;      // 16-byte units from `stats` to the end of `edge`
  float* S;               // [n_heads][L]  ranking score
  float* Su;              // [n_heads][L]  unpooled group-mean score (SnapKV layers, if wanted)
  float* edge;            // [n_heads][n_chunks][G][4 * pool_half] per-query-head A at chunk edges
  int32_t slot_layer[kMaxLayersPerLaunch];       // scored slot -> layer index in this group
  int32_t unscored_layer[kMaxLayersPerLaunch];   // unscored layer list
};

static_assert(sizeof(PrefillLaunch) <= 4000, "kernel argument block too large");

// Workspace layout for one launch group.
struct PrefillWorkspace {
  size_t counters, stats, S, Su, edge, end, total;
};

PrefillWorkspace prefill_workspace_layout(int n_heads, int n_chunks, int rows, int seq_len, int group,
                                          int pool_half, bool want_unpooled);

// Error reporting (thread-local last error).
int fail(int status, const std::string& msg);
void clear_error();

// Kernel launchers (prefill.hip / decode.hip).  Return a hipError_t as int.
int launch_prefill(const PrefillLaunch& P, int row_tiles, void* stream);

struct DecodeLayer {
  uint16_t* k_cache; uint16_t* v_cache; int32_t* pos; float* acc;
  const uint16_t* q; const uint16_t* k; const uint16_t* v; int32_t* victim;
  int32_t rule, capacity, recent;
  int32_t pad;
};

struct DecodeLaunch {
  DecodeLayer layer[kMaxLayersPerLaunch];
  int32_t n_layers, batch, n_q_heads, n_kv_heads, group, position, n_sink;
  float scale_log2;
};

static_assert(sizeof(DecodeLaunch) <= 4000, "kernel argument block too large");

int launch_decode(const DecodeLaunch& D, int max_capacity, void* stream);

// Stage timing with HIP events (enabled through rkv_profile_enable).
enum Stage { kStageZero = 0, kStageScore = 1, kStageSelect = 2, kStageGather = 3, kStageDecode = 4 };
void profile_mark(int stage, bool end, void* stream);

}  // namespace rkv

struct rkv_plan {
  std::vector<rkv_layer> layers;
  rkv_params params;
};
