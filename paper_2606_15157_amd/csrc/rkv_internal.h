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
constexpr int kSlice = 128;        // keys per scoring work item (4 waves x one tile of 32)
constexpr int kMaxRowTiles = 8;    // G * ceil(w / 32) supported by the scoring kernel
constexpr int kMaxPoolHalf = 64;   // pool_kernel / 2 supported
constexpr int kGatherRows = 32;    // retained rows per gather work item (one workgroup each)
constexpr int kCounterStride = 32; // words between per-job counters (one 128-byte line each)

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

// One prefill launch group (up to 32 layers).  A scored "job" is a (scored layer slot,
// sequence, KV head) triple, job = (slot * B + b) * Hkv + h; its keys are cut into n_slices
// slices of kSlice keys, the scoring work items.  The scored layers come first in `layer`
// (window-scored ones, then H2O with full-span accumulation, then TOVA), so slot s is layer[s]
// (slot_layer[s] == s).
struct PrefillLaunch {
  PrefillLayer layer[kMaxLayersPerLaunch];
  int32_t n_layers;
  int32_t n_scored;       // scored layer slots
  int32_t n_window;       // window-scored slots 0 .. n_window-1
  int32_t n_full;         // full-span H2O slots n_window .. n_window+n_full-1; TOVA slots follow
  int32_t n_gather;       // layers with retained rows (gather list)
  int32_t first_group;    // 1 in the call's first launch group: its first kernel clears the status word
  int32_t batch, seq_len, n_q_heads, n_kv_heads, window;
  int32_t group;          // G = Hq / Hkv
  int32_t row_tiles_per_group;  // ceil(w / 32)
  int32_t n_slices;       // ceil(L / kSlice)
  int32_t pool_half;      // pool_kernel / 2
  int32_t want_unpooled;  // write the unpooled group-mean score (acc seeding of SnapKV layers)
  float scale_log2;       // log2(e) / sqrt(d)
  int32_t force_window;   // test hook: the window kernels even where the pipelined one applies
  int32_t window_parts;   // window rows kernel: workgroups (key ranges) per job
  // workspace regions
  uint32_t* counters;     // [0] status; job j's slice-arrival counter at [kCounterStride * (1 + j)]
  float* stats;           // [J][n_slices][128]  pipelined kernel: per-slice row sums (NaN until stored);
                          // [J][window_parts][R]  window kernels with several parts: partial row sums
  float* part;            // [J][kPipeGroups][128]  pipelined kernel: per-group sums of those (NaN until stored)
  float* lam;             // [J][R]  window kernels: per-row log2 softmax normaliser (+inf for padding rows)
  float* ncl;             // [J][128]  pipelined kernel: minus the per-row reference logit (0 for padding rows);
                          // [J][R]  window kernels with several parts: the reference in log2 units (+inf: padding)
  float* lamf;            // [J_full][G][L]  full-span H2O: log2 normaliser of every query row
  float* tz;              // [J_tova][G][L]  TOVA: log2-scaled logits of the last query per head
  float* tstat;           // [J_tova][n_slices][G][2]  TOVA: per-slice (max, sum of exp2(x - max))
  float* S;               // [J][L]  ranking score
  float* Su;              // [J][L]  unpooled group-mean score (SnapKV layers, if wanted)
  float* edge;            // [J][n_slices][G][4 * pool_half]  per-query-head column sums at slice edges
  int32_t slot_layer[kMaxLayersPerLaunch];     // scored slot -> layer index in this group
  int32_t gather_layer[kMaxLayersPerLaunch];   // layers with retained rows
  int32_t gather_item0[kMaxLayersPerLaunch + 1];  // first gather work item of each gather layer (prefix)
};

static_assert(sizeof(PrefillLaunch) <= 4000, "kernel argument block too large");

// Workspace layout for one launch group.
struct PrefillWorkspace {
  size_t counters, stats, part, lam, ncl, lamf, tz, tstat, S, Su, edge, end, total;
};
PrefillWorkspace prefill_workspace_layout(int n_jobs, int n_slices, int rows, int seq_len, int group, int pool_half,
                                          int n_full_jobs, int n_tova_jobs);
constexpr int kPipeRows = 128;      // window rows of a job in the pipelined scoring kernel
constexpr int kPipeMaxSlices = 64;  // slices per job it takes
constexpr int kPipeGroups = 8;      // slice groups per job of its two-level row-sum exchange

// Key ranges per job of the window rows kernel: with few jobs, enough workgroups to fill the
// chip (two resident per CU at four row tiles, one at eight); at most 8 parts of at least 8
// slices each.  The host's workspace layout and launch both take it from here.
inline int window_parts(int n_window_jobs, int n_slices, int rows) {
  if (n_window_jobs <= 0) return 1;
  const int want = rows <= 4 * 32 ? 512 : 256;
  int p = (want + n_window_jobs - 1) / n_window_jobs;
  p = p < 8 ? p : 8;
  const int by_len = n_slices / 8 > 1 ? n_slices / 8 : 1;
  p = p < by_len ? p : by_len;
  return p > 1 ? p : 1;
}

// Error reporting (thread-local last error).
int fail(int status, const std::string& msg);
void clear_error();

// Kernel launchers (prefill.hip / decode.hip).  Return a hipError_t as int.
int launch_prefill(const PrefillLaunch& P, int row_tiles, void* stream);
int launch_fullspan(const PrefillLaunch& P, void* stream);   // fullspan.hip
int launch_tova(const PrefillLaunch& P, void* stream);       // tova.hip
int launch_window(const PrefillLaunch& P, int row_tiles, void* stream);   // window.hip

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

// Attention-entropy layer score (entropy.hip): up to kMaxLayersPerLaunch layers per launch.
struct EntropyLaunch {
  const uint16_t* q[kMaxLayersPerLaunch];   // [B, Hq, n_q, d]: positions L - n_q .. L - 1
  const uint16_t* k[kMaxLayersPerLaunch];   // [B, Hkv, L, d]
  int32_t n_layers, batch, seq_len, n_q_heads, n_kv_heads, n_q;
  float scale_log2;
  float* rows;        // [n_layers, B, Hq, n_q] row entropies (nats)
  float* h;           // [n_layers] mean row entropy
  double* partial;    // [n_layers, B * Hkv * ceil(n_q / 32)] per-workgroup sums of row entropies
  uint32_t* status;   // bit 0: some row entropy is not finite; bit 2: a block was recomputed exactly
  int32_t first_group;  // 1 in the call's first launch: it clears the status word
};

int launch_entropy(const EntropyLaunch& E, void* stream);

// Prefill -> decode hand-off (handoff.hip): up to kMaxCopies buffer copies per launch; a null
// source zero-fills the destination.  Sizes are in bytes, multiples of 4.
constexpr int kMaxCopies = 4 * kMaxLayersPerLaunch;
struct CopyTask {
  const void* src;
  void* dst;
  int64_t bytes;
};
struct CopyLaunch {
  CopyTask task[kMaxCopies];
  int32_t n_tasks;
};
static_assert(sizeof(CopyLaunch) <= 4000, "kernel argument block too large");
int launch_copies(const CopyLaunch& C, void* stream);

// Stage timing with HIP events (enabled through rkv_profile_enable).
enum Stage { kStageZero = 0, kStageScore = 1, kStageSelect = 2, kStageGather = 3, kStageDecode = 4 };
void profile_mark(int stage, bool end, void* stream);
// For a stage that is one kernel launch: when the stage is being profiled, two new events the
// launch records its start and stop in (hipExtLaunchKernelGGL: the dispatch's own timestamps,
// without the gaps that events recorded around it add); false otherwise.
bool profile_kernel_events(int stage, void** start, void** stop);

}  // namespace rkv

struct rkv_plan {
  std::vector<rkv_layer> layers;
  rkv_params params;
};
