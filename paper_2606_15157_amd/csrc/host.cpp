// Host side of librkv: errors, the capacity allocator, plan validation, argument
// checking, workspace layout and launch orchestration.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <mutex>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <new>
#include <numeric>

#include "rkv_internal.h"

namespace {
thread_local std::string g_error;

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool rule_valid(int32_t r) { return r >= RKV_FULL && r <= RKV_H2O_FULL; }

// The phases each operator's adapter declares (Section 3.4): bit 0 prefill, bit 1 decode.
// SnapKV and full-span H2O rank prompt positions by prompt queries, so they compress the prompt
// only; the others also have an incremental-update handler.
int32_t rule_phase_mask(int32_t r) {
  switch (r) {
    case RKV_SNAPKV:
    case RKV_H2O_FULL: return 1;
    case RKV_FULL:
    case RKV_STREAMING:
    case RKV_H2O:
    case RKV_TOVA: return 3;
    default: return 0;
  }
}
constexpr int32_t kPlanMagic = 0x50564b52;   // "RKVP" as little-endian bytes
constexpr int32_t kPlanFormat = 1;

// Retained positions and selection layout of one layer (prefill phase).
struct Layout {
  int32_t n_keep, cand_end, k_sel, forced_lo, forced_hi, all, scored;
};

// `want_scores`: the caller asked for score_out / acc_out of this layer.  A scoring rule is
// scored when it has to rank candidates or when its scores are an output.
Layout prefill_layout(const rkv_layer& ly, const rkv_params& p, int32_t L, bool want_scores = true) {
  Layout o{};
  const int32_t b = ly.budget_prefill;
  o.scored = (ly.rule_prefill == RKV_SNAPKV || ly.rule_prefill == RKV_H2O || ly.rule_prefill == RKV_H2O_FULL ||
              ly.rule_prefill == RKV_TOVA) ? 1 : 0;
  if (ly.rule_prefill == RKV_FULL || b >= L) {
    o.n_keep = L; o.all = 1; o.cand_end = 0; o.k_sel = 0; o.forced_lo = 0; o.forced_hi = L;
    if (o.scored && !want_scores) o.scored = 0;
    return o;
  }
  o.n_keep = b;
  switch (ly.rule_prefill) {
    case RKV_STREAMING: {
      int32_t s0 = std::min(p.n_sink, b);
      o.cand_end = s0; o.k_sel = s0; o.forced_lo = L - (b - s0); o.forced_hi = L;
      break;
    }
    case RKV_SNAPKV:
      if (b <= p.window) { o.cand_end = 0; o.k_sel = 0; o.forced_lo = L - b; }
      else { o.cand_end = L - p.window; o.k_sel = b - p.window; o.forced_lo = L - p.window; }
      o.forced_hi = L;
      break;
    case RKV_H2O:
    case RKV_H2O_FULL: {
      int32_t r = (int32_t)(((int64_t)b * p.recent_num) / p.recent_den);
      o.cand_end = L - r; o.k_sel = b - r; o.forced_lo = L - r; o.forced_hi = L;
      break;
    }
    case RKV_TOVA:
      // every position is a candidate, nothing is forced
      o.cand_end = L; o.k_sel = b; o.forced_lo = L; o.forced_hi = L;
      break;
    default: break;
  }
  if (o.scored && o.k_sel == 0 && !want_scores) o.scored = 0;
  return o;
}

int validate_shape(const rkv_shape* s) {
  if (!s) return rkv::fail(RKV_ERR_INVALID_ARG, "shape is null");
  if (s->batch < 1 || s->seq_len < 1 || s->n_q_heads < 1 || s->n_kv_heads < 1 || s->head_dim < 1)
    return rkv::fail(RKV_ERR_SHAPE, "shape fields must be positive");
  if (s->n_q_heads % s->n_kv_heads)
    return rkv::fail(RKV_ERR_SHAPE, "n_q_heads must be a multiple of n_kv_heads");
  if (s->head_dim != rkv::kHeadDim)
    return rkv::fail(RKV_ERR_UNSUPPORTED, "head_dim must be 128");
  if (s->seq_len > (1 << 24)) return rkv::fail(RKV_ERR_UNSUPPORTED, "seq_len above 2^24");
  return RKV_OK;
}

int row_tiles(const rkv_params& p, const rkv_shape* s) {
  int G = s->n_q_heads / s->n_kv_heads;
  return G * ((p.window + 31) / 32);
}

// Scoring row tiles padded to a supported kernel instantiation (4 or 8 tiles of 32 rows).
int kernel_row_tiles(int nt) { return nt <= 4 ? 4 : 8; }

struct Group {
  int l0, l1, n_scored, n_full, n_tova;   // scored layers; of which full-span H2O, TOVA
};

// Scoring class of a layer in a launch group: 0 window-scored, 1 full-span H2O, 2 TOVA,
// 3 not scored.  Slots follow this order.
int score_class(const rkv_layer& ly, const Layout& lo) {
  if (!lo.scored) return 3;
  if (ly.rule_prefill == RKV_H2O_FULL) return 1;
  if (ly.rule_prefill == RKV_TOVA) return 2;
  return 0;
}

// Test hook: RKV_FORCE_WINDOW=1 selects the window scoring kernels (normally used for prompts of
// more than 64 slices and for eight row tiles) on layouts the pipelined kernel would take, so
// that they can be checked on short prompts too.
int force_window() {
  const char* e = std::getenv("RKV_FORCE_WINDOW");
  return e && std::atoi(e) > 0 ? 1 : 0;
}

std::vector<Group> layer_groups(const rkv_plan* plan, int32_t L) {
  std::vector<Group> g;
  int n = (int)plan->layers.size();
  for (int l0 = 0; l0 < n; l0 += rkv::kMaxLayersPerLaunch) {
    int l1 = std::min(n, l0 + rkv::kMaxLayersPerLaunch);
    int sc = 0, nf = 0, nt = 0;
    for (int l = l0; l < l1; ++l) {
      const int cls = score_class(plan->layers[l], prefill_layout(plan->layers[l], plan->params, L));
      sc += cls < 3;
      nf += cls == 1;
      nt += cls == 2;
    }
    g.push_back({l0, l1, sc, nf, nt});
  }
  return g;
}

size_t group_workspace(const rkv_plan* plan, const rkv_shape* s, const Group& g) {
  const int L = s->seq_len;
  const int G = s->n_q_heads / s->n_kv_heads;
  const int nt = kernel_row_tiles(row_tiles(plan->params, s));
  const int n_jobs = s->batch * g.n_scored * s->n_kv_heads;
  const int n_slices = (L + rkv::kSlice - 1) / rkv::kSlice;
  return rkv::prefill_workspace_layout(n_jobs, n_slices, nt * 32, L, G, plan->params.pool_kernel / 2,
                                       s->batch * g.n_full * s->n_kv_heads,
                                       s->batch * g.n_tova * s->n_kv_heads).total;
}

}  // namespace

namespace rkv {

namespace {
std::mutex g_prof_mu;
int g_prof_stage = -1;
std::vector<hipEvent_t> g_prof_events;  // begin/end pairs
std::vector<hipEvent_t> g_prof_pool;    // created events not in use (taken by the marks, returned by the read)
constexpr size_t kMaxProfiled = 4096;
// Profiling events skip the system-scope memory fence of an ordinary event record (the kernels
// they bracket need no fence to be timed).
constexpr unsigned kProfEventFlags = hipEventDisableSystemFence;
constexpr size_t kProfPoolFill = 1024;   // events created when profiling is enabled

// An event from the pool (created on demand when the pool is empty); g_prof_mu held.
bool take_event(hipEvent_t* e) {
  if (!g_prof_pool.empty()) {
    *e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return true;
  }
  return hipEventCreateWithFlags(e, kProfEventFlags) == hipSuccess;
}
}  // namespace

void profile_mark(int stage, bool end, void* stream) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (stage != g_prof_stage) return;
  if (!end && g_prof_events.size() >= 2 * kMaxProfiled) return;
  if (end && g_prof_events.size() % 2 == 0) return;  // begin was dropped
  hipEvent_t e;
  if (!take_event(&e)) return;
  if (hipEventRecord(e, reinterpret_cast<hipStream_t>(stream)) != hipSuccess) {
    g_prof_pool.push_back(e);
    return;
  }
  g_prof_events.push_back(e);
}

bool profile_kernel_events(int stage, void** start, void** stop) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  *start = *stop = nullptr;
  if (stage != g_prof_stage || g_prof_events.size() % 2 != 0 || g_prof_events.size() >= 2 * kMaxProfiled) return false;
  hipEvent_t a, b;
  if (!take_event(&a)) return false;
  if (!take_event(&b)) {
    g_prof_pool.push_back(a);
    return false;
  }
  g_prof_events.push_back(a);
  g_prof_events.push_back(b);
  *start = a;
  *stop = b;
  return true;
}

int fail(int status, const std::string& msg) {
  g_error = msg;
  return status;
}

void clear_error() { g_error.clear(); }

PrefillWorkspace prefill_workspace_layout(int n_jobs, int n_slices, int rows, int seq_len, int group, int pool_half,
                                          int n_full_jobs, int n_tova_jobs) {
  PrefillWorkspace w{};
  size_t off = 0;
  w.counters = off;
  off = round_up(off + sizeof(uint32_t) * kCounterStride * (1 + (size_t)n_jobs), 256);
  // per-slice row sums of the pipelined kernel (four row tiles, at most kPipeMaxSlices slices), or
  // the window rows kernel's partial row sums; the first is never smaller where both could run
  w.stats = off;
  const bool pipe_layout = rows == kPipeRows && n_slices <= kPipeMaxSlices;
  const int parts = window_parts(n_jobs - n_full_jobs - n_tova_jobs, n_slices, rows);
  const size_t stat_floats = pipe_layout ? (size_t)n_jobs * n_slices * kPipeRows
                                         : (parts > 1 ? (size_t)n_jobs * parts * rows : 0);
  off = round_up(off + sizeof(float) * stat_floats, 256);
  // the pipelined kernel's per-group sums of the row sums
  w.part = off;
  off = round_up(off + sizeof(float) * (pipe_layout ? (size_t)n_jobs * kPipeGroups * kPipeRows : 0), 256);
  w.lam = off;
  off = round_up(off + sizeof(float) * (size_t)n_jobs * rows, 256);
  w.ncl = off;
  off = round_up(off + sizeof(float) * (size_t)n_jobs * rows, 256);
  w.lamf = off;
  off = round_up(off + sizeof(float) * (size_t)n_full_jobs * group * seq_len, 256);
  w.tz = off;
  off = round_up(off + sizeof(float) * (size_t)n_tova_jobs * group * seq_len, 256);
  w.tstat = off;
  off = round_up(off + sizeof(float) * 2 * (size_t)n_tova_jobs * n_slices * group, 256);
  w.S = off;
  off = round_up(off + sizeof(float) * (size_t)n_jobs * seq_len, 256);
  w.Su = off;
  off = round_up(off + sizeof(float) * (size_t)n_jobs * seq_len, 256);
  w.edge = off;
  off = round_up(off + sizeof(float) * (size_t)n_jobs * n_slices * group * 4 * std::max(pool_half, 1), 256);
  w.end = off;
  w.total = std::max<size_t>(off, 256);
  return w;
}

}  // namespace rkv

extern "C" {

const char* rkv_last_error(void) { return g_error.c_str(); }

int rkv_profile_enable(int32_t stage) {
  rkv::clear_error();
  if (stage < -1 || stage > rkv::kStageDecode) return rkv::fail(RKV_ERR_INVALID_ARG, "unknown stage");
  std::lock_guard<std::mutex> lk(rkv::g_prof_mu);
  rkv::g_prof_stage = stage;
  // create the events up front: creating them during the profiled launches would slow the host
  // enough to leave the GPU idle between launches
  while (stage >= 0 && rkv::g_prof_pool.size() + rkv::g_prof_events.size() < rkv::kProfPoolFill) {
    hipEvent_t e;
    if (hipEventCreateWithFlags(&e, rkv::kProfEventFlags) != hipSuccess) break;
    rkv::g_prof_pool.push_back(e);
  }
  return RKV_OK;
}

int rkv_profile_read(int32_t* n_launches, double* total_ms) {
  rkv::clear_error();
  if (!n_launches || !total_ms) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  std::lock_guard<std::mutex> lk(rkv::g_prof_mu);
  std::vector<hipEvent_t>& ev = rkv::g_prof_events;
  double tot = 0.0;
  int n = 0;
  int st = RKV_OK;
  for (size_t i = 0; i + 1 < ev.size(); i += 2) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(ev[i + 1]);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev[i], ev[i + 1]);
    if (e != hipSuccess) {
      st = rkv::fail(RKV_ERR_HIP, std::string("event timing: ") + hipGetErrorString(e));
      break;
    }
    tot += ms;
    ++n;
  }
  for (hipEvent_t e : ev) rkv::g_prof_pool.push_back(e);   // reused by later profiled launches
  ev.clear();
  *n_launches = n;
  *total_ms = tot;
  return st;
}

int rkv_version(void) { return RKV_VERSION; }

int rkv_allocate_budgets(const double* scores, int32_t n_layers, int32_t transform, int64_t total,
                         int32_t b_min, int32_t* budgets_out) {
  rkv::clear_error();
  if (!scores || !budgets_out) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  if (n_layers < 1) return rkv::fail(RKV_ERR_INVALID_ARG, "n_layers must be >= 1");
  if (b_min < 0) return rkv::fail(RKV_ERR_INVALID_ARG, "b_min must be >= 0");
  if (total < (int64_t)n_layers * b_min) return rkv::fail(RKV_ERR_INVALID_ARG, "total below n_layers * b_min");
  if (total > ((int64_t)1 << 40)) return rkv::fail(RKV_ERR_INVALID_ARG, "total too large");
  if (transform != RKV_T_IDENTITY && transform != RKV_T_PPL_CAP)
    return rkv::fail(RKV_ERR_INVALID_ARG, "unknown transform");
  const int n = n_layers;
  std::vector<double> t(scores, scores + n);
  for (double x : t)
    if (!std::isfinite(x)) return rkv::fail(RKV_ERR_INVALID_ARG, "scores must be finite");
  if (transform == RKV_T_PPL_CAP) {
    // 95th percentile by linear interpolation between order statistics
    std::vector<double> srt(t);
    std::sort(srt.begin(), srt.end());
    double rank = 0.95 * (n - 1);
    int lo = (int)std::floor(rank);
    int hi = std::min(lo + 1, n - 1);
    double cap = srt[lo] + (rank - lo) * (srt[hi] - srt[lo]);
    for (double& x : t) x = std::min(x, cap);
  }
  double mn = *std::min_element(t.begin(), t.end());
  if (mn <= 0.0)
    for (double& x : t) x = x - mn + 1e-6;
  // provisional shares with the iterative b_min clamp
  std::vector<char> fixed(n, 0);
  std::vector<double> share(n, 0.0);
  for (;;) {
    double wsum = 0.0;
    int nfixed = 0;
    for (int i = 0; i < n; ++i) {
      if (fixed[i]) ++nfixed; else wsum += t[i];
    }
    double remaining = (double)total - (double)b_min * nfixed;
    bool added = false;
    for (int i = 0; i < n; ++i) {
      if (fixed[i]) { share[i] = b_min; continue; }
      share[i] = remaining * t[i] / wsum;
    }
    for (int i = 0; i < n; ++i)
      if (!fixed[i] && share[i] < b_min) { fixed[i] = 1; added = true; }
    if (!added) break;
  }
  // floor, then the residual to the largest fractional remainders (ties: lower layer)
  std::vector<int64_t> base(n);
  std::vector<double> frac(n);
  int64_t sum = 0;
  for (int i = 0; i < n; ++i) {
    base[i] = (int64_t)std::floor(share[i]);
    frac[i] = share[i] - (double)base[i];
    sum += base[i];
  }
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return frac[a] > frac[b]; });
  int64_t residual = total - sum;
  for (int64_t r = 0; r < residual && r < n; ++r) base[order[r]] += 1;
  for (int i = 0; i < n; ++i) {
    if (base[i] > INT32_MAX) return rkv::fail(RKV_ERR_INVALID_ARG, "budget overflows int32");
  }
  for (int i = 0; i < n; ++i) budgets_out[i] = (int32_t)base[i];
  return RKV_OK;
}

int rkv_plan_create(const rkv_layer* layers, int32_t n_layers, const rkv_params* params, rkv_plan** out) {
  rkv::clear_error();
  if (!layers || !params || !out) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  if (n_layers < 1) return rkv::fail(RKV_ERR_INVALID_ARG, "n_layers must be >= 1");
  const rkv_params& p = *params;
  if (p.window < 1) return rkv::fail(RKV_ERR_PLAN, "window must be >= 1");
  if (p.pool_kernel < 1 || p.pool_kernel % 2 == 0) return rkv::fail(RKV_ERR_PLAN, "pool_kernel must be odd and >= 1");
  if (p.pool_kernel / 2 > rkv::kMaxPoolHalf) return rkv::fail(RKV_ERR_UNSUPPORTED, "pool_kernel above 129");
  if (p.n_sink < 0) return rkv::fail(RKV_ERR_PLAN, "n_sink must be >= 0");
  if (p.recent_den < 1 || p.recent_num < 0 || p.recent_num > p.recent_den)
    return rkv::fail(RKV_ERR_PLAN, "need 0 <= recent_num <= recent_den, recent_den >= 1");
  for (int l = 0; l < n_layers; ++l) {
    const rkv_layer& ly = layers[l];
    if (!rule_valid(ly.rule_prefill) || !rule_valid(ly.rule_decode))
      return rkv::fail(RKV_ERR_INVALID_ARG, "layer " + std::to_string(l) + ": unknown rule");
    if (ly.budget_prefill < 0 || ly.budget_decode < 0)
      return rkv::fail(RKV_ERR_PLAN, "layer " + std::to_string(l) + ": negative budget");
    if (!(rule_phase_mask(ly.rule_prefill) & 1))
      return rkv::fail(RKV_ERR_PLAN, "layer " + std::to_string(l) + ": operator not declared for prefill");
    if (ly.rule_decode == RKV_SNAPKV)
      return rkv::fail(RKV_ERR_PLAN, "layer " + std::to_string(l) + ": SnapKV compresses the prompt only, not valid in decode");
    if (ly.rule_decode == RKV_H2O_FULL)
      return rkv::fail(RKV_ERR_PLAN, "layer " + std::to_string(l) + ": full-span accumulation is a prefill rule (decode uses RKV_H2O)");
    if (ly.rule_decode == RKV_TOVA && ly.budget_decode < 1)
      return rkv::fail(RKV_ERR_PLAN, "layer " + std::to_string(l) + ": decode TOVA needs budget >= 1");
    if (ly.rule_decode == RKV_H2O && ly.budget_decode < 2)
      return rkv::fail(RKV_ERR_PLAN, "layer " + std::to_string(l) + ": decode H2O needs budget >= 2");
    if (ly.rule_decode == RKV_STREAMING && ly.budget_decode < 1)
      return rkv::fail(RKV_ERR_PLAN, "layer " + std::to_string(l) + ": decode StreamingLLM needs budget >= 1");
  }
  rkv_plan* plan = new (std::nothrow) rkv_plan;
  if (!plan) return rkv::fail(RKV_ERR_INVALID_ARG, "out of host memory");
  plan->layers.assign(layers, layers + n_layers);
  plan->params = p;
  *out = plan;
  return RKV_OK;
}

int rkv_rule_phases(int32_t rule, int32_t* phase_mask) {
  rkv::clear_error();
  if (!phase_mask) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  if (!rule_valid(rule)) return rkv::fail(RKV_ERR_INVALID_ARG, "unknown rule");
  *phase_mask = rule_phase_mask(rule);
  return RKV_OK;
}

int rkv_plan_from_route(const rkv_route_layer* route, int32_t n_layers, const rkv_params* params, rkv_plan** out) {
  rkv::clear_error();
  if (!route || !params || !out) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  if (n_layers < 1) return rkv::fail(RKV_ERR_INVALID_ARG, "n_layers must be >= 1");
  std::vector<rkv_layer> layers((size_t)n_layers);
  for (int l = 0; l < n_layers; ++l) {
    const rkv_route_layer& r = route[l];
    const std::string at = "layer " + std::to_string(l) + ": ";
    if (!rule_valid(r.rule)) return rkv::fail(RKV_ERR_INVALID_ARG, at + "unknown rule");
    if (r.scope < RKV_SCOPE_PREFILL || r.scope > RKV_SCOPE_BOTH) return rkv::fail(RKV_ERR_INVALID_ARG, at + "unknown scope");
    // the phases the scope activates must all be declared by the operator (for BOTH: the
    // intersection of the prefill and decode declarations)
    const int32_t need = r.scope == RKV_SCOPE_PREFILL ? 1 : (r.scope == RKV_SCOPE_DECODE ? 2 : 3);
    if ((rule_phase_mask(r.rule) & need) != need)
      return rkv::fail(RKV_ERR_PLAN, at + (r.scope == RKV_SCOPE_BOTH
                                               ? "a tied both-phase route needs an operator declared for both phases"
                                               : "operator not declared for the scope's phase"));
    const bool pre = need & 1, dec = need & 2;
    layers[l].rule_prefill = pre ? r.rule : RKV_FULL;
    layers[l].budget_prefill = pre ? r.budget : 0;
    layers[l].rule_decode = dec ? r.rule : RKV_FULL;
    layers[l].budget_decode = dec ? r.budget : 0;
  }
  return rkv_plan_create(layers.data(), n_layers, params, out);
}

void rkv_plan_destroy(rkv_plan* plan) { delete plan; }

int rkv_plan_serialize(const rkv_plan* plan, void* buf, size_t cap, size_t* size) {
  rkv::clear_error();
  if (!plan || !size) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  const size_t n = plan->layers.size();
  const size_t need = 32 + 16 * n;
  *size = need;
  if (!buf) return RKV_OK;
  if (cap < need) return rkv::fail(RKV_ERR_INVALID_ARG, "buffer too small for the serialized plan");
  std::vector<int32_t> w;
  w.reserve(need / 4);
  w.push_back(kPlanMagic);
  w.push_back(kPlanFormat);
  w.push_back((int32_t)n);
  const rkv_params& p = plan->params;
  for (int32_t v : {p.window, p.pool_kernel, p.n_sink, p.recent_num, p.recent_den}) w.push_back(v);
  for (const rkv_layer& ly : plan->layers)
    for (int32_t v : {ly.rule_prefill, ly.budget_prefill, ly.rule_decode, ly.budget_decode}) w.push_back(v);
  unsigned char* o = static_cast<unsigned char*>(buf);
  for (size_t i = 0; i < w.size(); ++i) {   // little-endian, independent of the host's byte order
    const uint32_t u = (uint32_t)w[i];
    for (int b = 0; b < 4; ++b) o[4 * i + b] = (unsigned char)(u >> (8 * b));
  }
  return RKV_OK;
}

int rkv_plan_deserialize(const void* buf, size_t size, rkv_plan** out) {
  rkv::clear_error();
  if (!buf || !out) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  if (size < 32 || size % 4) return rkv::fail(RKV_ERR_INVALID_ARG, "serialized plan has a bad length");
  const unsigned char* in = static_cast<const unsigned char*>(buf);
  auto word = [&](size_t i) {
    uint32_t u = 0;
    for (int b = 0; b < 4; ++b) u |= (uint32_t)in[4 * i + b] << (8 * b);
    return (int32_t)u;
  };
  if (word(0) != kPlanMagic) return rkv::fail(RKV_ERR_INVALID_ARG, "not a serialized plan (magic)");
  if (word(1) != kPlanFormat) return rkv::fail(RKV_ERR_INVALID_ARG, "unknown serialized plan format version");
  const int32_t n = word(2);
  if (n < 1 || size != 32 + 16 * (size_t)n) return rkv::fail(RKV_ERR_INVALID_ARG, "serialized plan length does not match its layer count");
  rkv_params p;
  p.window = word(3);
  p.pool_kernel = word(4);
  p.n_sink = word(5);
  p.recent_num = word(6);
  p.recent_den = word(7);
  std::vector<rkv_layer> layers((size_t)n);
  for (int32_t l = 0; l < n; ++l) {
    layers[l].rule_prefill = word(8 + 4 * l);
    layers[l].budget_prefill = word(9 + 4 * l);
    layers[l].rule_decode = word(10 + 4 * l);
    layers[l].budget_decode = word(11 + 4 * l);
  }
  return rkv_plan_create(layers.data(), n, &p, out);
}

int rkv_plan_num_layers(const rkv_plan* plan, int32_t* n_layers) {
  rkv::clear_error();
  if (!plan || !n_layers) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  *n_layers = (int32_t)plan->layers.size();
  return RKV_OK;
}

int rkv_plan_retained_counts(const rkv_plan* plan, int32_t phase, int32_t seq_len, int32_t* counts_out) {
  rkv::clear_error();
  if (!plan || !counts_out) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  if (phase != RKV_PHASE_PREFILL && phase != RKV_PHASE_DECODE) return rkv::fail(RKV_ERR_INVALID_ARG, "unknown phase");
  if (seq_len < 0) return rkv::fail(RKV_ERR_INVALID_ARG, "seq_len must be >= 0");
  for (size_t l = 0; l < plan->layers.size(); ++l) {
    const rkv_layer& ly = plan->layers[l];
    int32_t rule = phase == RKV_PHASE_PREFILL ? ly.rule_prefill : ly.rule_decode;
    int32_t b = phase == RKV_PHASE_PREFILL ? ly.budget_prefill : ly.budget_decode;
    counts_out[l] = rule == RKV_FULL ? seq_len : std::min(b, seq_len);
  }
  return RKV_OK;
}

int rkv_prefill_workspace_size(const rkv_plan* plan, const rkv_shape* shape, size_t* bytes) {
  rkv::clear_error();
  if (!plan || !bytes) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  int st = validate_shape(shape);
  if (st) return st;
  size_t need = 256;
  for (const Group& g : layer_groups(plan, shape->seq_len)) need = std::max(need, group_workspace(plan, shape, g));
  *bytes = need;
  return RKV_OK;
}

int rkv_prefill_evict(const rkv_plan* plan, const rkv_shape* shape, const rkv_prefill_io* io, void* ws,
                      size_t ws_bytes, void* stream) {
  rkv::clear_error();
  if (!plan || !io) return rkv::fail(RKV_ERR_INVALID_ARG, "null plan or io");
  int st = validate_shape(shape);
  if (st) return st;
  const rkv_params& p = plan->params;
  const int L = shape->seq_len;
  if (p.window > L) return rkv::fail(RKV_ERR_SHAPE, "window larger than seq_len");
  if (!io->k || !io->v || !io->k_out || !io->v_out || !io->idx_out)
    return rkv::fail(RKV_ERR_INVALID_ARG, "io arrays k, v, k_out, v_out, idx_out are required");
  const int n = (int)plan->layers.size();
  const int G = shape->n_q_heads / shape->n_kv_heads;
  const int nt = row_tiles(p, shape);
  bool any_window = false, any_g_bound = false;
  for (int l = 0; l < n; ++l) {
    Layout lo = prefill_layout(plan->layers[l], p, L);
    const int cls = score_class(plan->layers[l], lo);
    any_window |= cls == 0;
    any_g_bound |= cls == 1 || cls == 2;
    if (!io->k[l] || !io->v[l]) return rkv::fail(RKV_ERR_INVALID_ARG, "layer " + std::to_string(l) + ": null k or v");
    if (!io->k_out[l] || !io->v_out[l] || !io->idx_out[l])
      if (lo.n_keep > 0) return rkv::fail(RKV_ERR_INVALID_ARG, "layer " + std::to_string(l) + ": null output");
    if (lo.scored && (!io->q_win || !io->q_win[l]))
      return rkv::fail(RKV_ERR_INVALID_ARG, "layer " + std::to_string(l) + ": scoring rule needs q_win");
  }
  if (any_window && nt > rkv::kMaxRowTiles)
    return rkv::fail(RKV_ERR_UNSUPPORTED, "G * ceil(window / 32) must be <= 8");
  if (any_g_bound && G != 1 && G != 2 && G != 4 && G != 8)
    return rkv::fail(RKV_ERR_UNSUPPORTED, "TOVA and full-span H2O layers need n_q_heads / n_kv_heads in {1, 2, 4, 8}");
  size_t need = 256;
  std::vector<Group> groups = layer_groups(plan, L);
  for (const Group& g : groups) need = std::max(need, group_workspace(plan, shape, g));
  if (!ws) return rkv::fail(RKV_ERR_WORKSPACE, "workspace is null");
  if (((uintptr_t)ws) % 256) return rkv::fail(RKV_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need)
    return rkv::fail(RKV_ERR_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes");

  const int ktiles = kernel_row_tiles(nt);
  bool first = true;
  for (const Group& g : groups) {
    rkv::PrefillLaunch P;
    std::memset(&P, 0, sizeof(P));
    P.first_group = first ? 1 : 0;
    first = false;
    P.n_layers = g.l1 - g.l0;
    P.batch = shape->batch;
    P.seq_len = L;
    P.n_q_heads = shape->n_q_heads;
    P.n_kv_heads = shape->n_kv_heads;
    P.window = p.window;
    P.group = G;
    P.row_tiles_per_group = (p.window + 31) / 32;
    P.n_slices = (L + rkv::kSlice - 1) / rkv::kSlice;
    P.pool_half = p.pool_kernel / 2;
    P.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)shape->head_dim));
    P.force_window = force_window();
    int slot = 0, n_gather = 0;
    bool want_unpooled = false;
    // scored layers first, so that scored slot s is entry s of the layer table (the pipelined
    // scoring kernel looks a slot's tensors up with one load)
    int order[rkv::kMaxLayersPerLaunch];
    Layout lays[rkv::kMaxLayersPerLaunch];
    int n_class[4] = {0, 0, 0, 0};
    {
      // window-scored layers, then full-span H2O, then TOVA, then the unscored ones
      int n = 0;
      for (int pass = 0; pass < 4; ++pass)
        for (int i = 0; i < P.n_layers; ++i) {
          const int l = g.l0 + i;
          const bool want = (io->score_out && io->score_out[l]) || (io->acc_out && io->acc_out[l]);
          const Layout lo = prefill_layout(plan->layers[l], p, L, want);
          if (score_class(plan->layers[l], lo) == pass) {
            lays[n] = lo;
            order[n++] = i;
            ++n_class[pass];
          }
        }
    }
    const int n_window = n_class[0];
    for (int i = 0; i < P.n_layers; ++i) {
      const int l = g.l0 + order[i];
      const Layout& lo = lays[i];
      rkv::PrefillLayer& d = P.layer[i];
      d.q = io->q_win ? (const uint16_t*)io->q_win[l] : nullptr;
      d.k = (const uint16_t*)io->k[l];
      d.v = (const uint16_t*)io->v[l];
      d.k_out = (uint16_t*)io->k_out[l];
      d.v_out = (uint16_t*)io->v_out[l];
      d.idx = io->idx_out[l];
      d.score = io->score_out ? io->score_out[l] : nullptr;
      d.acc = io->acc_out ? io->acc_out[l] : nullptr;
      d.rule = plan->layers[l].rule_prefill;
      d.n_keep = lo.n_keep;
      d.cand_end = lo.cand_end;
      d.k_sel = lo.k_sel;
      d.forced_lo = lo.forced_lo;
      d.forced_hi = lo.forced_hi;
      d.all = lo.all;
      d.slot = lo.scored ? slot : -1;
      if (lo.scored) {
        P.slot_layer[slot] = i;
        if (d.rule == RKV_SNAPKV && d.acc) want_unpooled = true;
        ++slot;
      }
      if (lo.n_keep > 0) P.gather_layer[n_gather++] = i;
    }
    P.n_scored = slot;
    P.n_window = n_window;
    P.n_full = n_class[1];
    P.n_gather = n_gather;
    P.gather_item0[0] = 0;
    for (int i = 0; i < n_gather; ++i) {
      const int64_t rows = (int64_t)shape->batch * shape->n_kv_heads * P.layer[P.gather_layer[i]].n_keep;
      P.gather_item0[i + 1] = P.gather_item0[i] + (int32_t)((rows + rkv::kGatherRows - 1) / rkv::kGatherRows);
    }
    P.want_unpooled = want_unpooled ? 1 : 0;
    const int n_jobs = shape->batch * slot * shape->n_kv_heads;
    const int n_full_jobs = shape->batch * n_class[1] * shape->n_kv_heads;
    const int n_tova_jobs = shape->batch * n_class[2] * shape->n_kv_heads;
    rkv::PrefillWorkspace W = rkv::prefill_workspace_layout(n_jobs, P.n_slices, ktiles * 32, L, G, P.pool_half,
                                                            n_full_jobs, n_tova_jobs);
    P.window_parts = rkv::window_parts(n_jobs - n_full_jobs - n_tova_jobs, P.n_slices, ktiles * 32);
    char* base = (char*)ws;
    P.counters = (uint32_t*)(base + W.counters);
    P.stats = (float*)(base + W.stats);
    P.part = (float*)(base + W.part);
    P.lam = (float*)(base + W.lam);
    P.ncl = (float*)(base + W.ncl);
    P.lamf = (float*)(base + W.lamf);
    P.tz = (float*)(base + W.tz);
    P.tstat = (float*)(base + W.tstat);
    P.S = (float*)(base + W.S);
    P.Su = (float*)(base + W.Su);
    P.edge = (float*)(base + W.edge);
    int err = rkv::launch_prefill(P, ktiles, stream);
    if (err) return rkv::fail(RKV_ERR_HIP, std::string("kernel launch failed: ") + hipGetErrorString((hipError_t)err));
  }
  return RKV_OK;
}

int rkv_prefill_check(const void* ws, size_t ws_bytes, int32_t* status_out) {
  rkv::clear_error();
  if (!ws || !status_out) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  if (ws_bytes < sizeof(uint32_t)) return rkv::fail(RKV_ERR_WORKSPACE, "workspace too small");
  uint32_t v = 0;
  hipError_t e = hipMemcpy(&v, ws, sizeof(v), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return rkv::fail(RKV_ERR_HIP, std::string("hipMemcpy: ") + hipGetErrorString(e));
  *status_out = (int32_t)v;
  return RKV_OK;
}

namespace {
size_t entropy_blocks_per_layer(const rkv_shape* s, int32_t n_q) {
  return (size_t)s->batch * s->n_kv_heads * (size_t)((n_q + 31) / 32);
}
}  // namespace

int rkv_entropy_workspace_size(const rkv_shape* shape, int32_t n_layers, int32_t n_q, size_t* bytes) {
  rkv::clear_error();
  if (!bytes) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  if (n_layers < 1) return rkv::fail(RKV_ERR_INVALID_ARG, "n_layers must be >= 1");
  int st = validate_shape(shape);
  if (st) return st;
  if (n_q < 1 || n_q > shape->seq_len) return rkv::fail(RKV_ERR_INVALID_ARG, "n_q must lie in [1, seq_len]");
  *bytes = sizeof(double) * (size_t)n_layers * entropy_blocks_per_layer(shape, n_q);
  return RKV_OK;
}

int rkv_entropy_profile(const rkv_shape* shape, int32_t n_layers, int32_t n_q, const void* const* q,
                        const void* const* k, float* rows_out, float* h_out, uint32_t* status, void* ws,
                        size_t ws_bytes, void* stream) {
  rkv::clear_error();
  if (!shape || !q || !k || !rows_out || !h_out || !status) return rkv::fail(RKV_ERR_INVALID_ARG, "null pointer");
  size_t need = 0;
  int st0 = rkv_entropy_workspace_size(shape, n_layers, n_q, &need);
  if (st0) return st0;
  if (!ws || ws_bytes < need || ((uintptr_t)ws & 7))
    return rkv::fail(RKV_ERR_WORKSPACE, "entropy workspace missing, too small or not 8-byte aligned");
  if (n_layers < 1) return rkv::fail(RKV_ERR_INVALID_ARG, "n_layers must be >= 1");
  int st = validate_shape(shape);
  if (st) return st;
  const int L = shape->seq_len;
  if (n_q < 1 || n_q > L) return rkv::fail(RKV_ERR_INVALID_ARG, "n_q must lie in [1, seq_len]");
  const int G = shape->n_q_heads / shape->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return rkv::fail(RKV_ERR_UNSUPPORTED, "entropy profile needs n_q_heads / n_kv_heads in {1, 2, 4, 8}");
  const size_t per_layer = (size_t)shape->batch * shape->n_q_heads * n_q;
  for (int l = 0; l < n_layers; ++l)
    if (!q[l] || !k[l]) return rkv::fail(RKV_ERR_INVALID_ARG, "layer " + std::to_string(l) + ": null q or k");
  for (int l0 = 0; l0 < n_layers; l0 += rkv::kMaxLayersPerLaunch) {
    rkv::EntropyLaunch E;
    std::memset(&E, 0, sizeof(E));
    E.n_layers = std::min(n_layers - l0, rkv::kMaxLayersPerLaunch);
    E.first_group = l0 == 0 ? 1 : 0;
    for (int i = 0; i < E.n_layers; ++i) {
      E.q[i] = (const uint16_t*)q[l0 + i];
      E.k[i] = (const uint16_t*)k[l0 + i];
    }
    E.batch = shape->batch;
    E.seq_len = L;
    E.n_q_heads = shape->n_q_heads;
    E.n_kv_heads = shape->n_kv_heads;
    E.n_q = n_q;
    E.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)shape->head_dim));
    E.rows = rows_out + (size_t)l0 * per_layer;
    E.h = h_out + l0;
    E.status = status;
    E.partial = static_cast<double*>(ws) + (size_t)l0 * entropy_blocks_per_layer(shape, n_q);
    int err = rkv::launch_entropy(E, stream);
    if (err) return rkv::fail(RKV_ERR_HIP, std::string("kernel launch failed: ") + hipGetErrorString((hipError_t)err));
  }
  return RKV_OK;
}

int rkv_decode_step(const rkv_plan* plan, const rkv_shape* shape, const rkv_decode_state* state,
                    const rkv_decode_input* input, int32_t position, void* stream) {
  rkv::clear_error();
  if (!plan || !state || !input) return rkv::fail(RKV_ERR_INVALID_ARG, "null plan, state or input");
  int st = validate_shape(shape);
  if (st) return st;
  if (!state->k_cache || !state->v_cache || !state->pos || !input->q || !input->k || !input->v)
    return rkv::fail(RKV_ERR_INVALID_ARG, "state and input arrays are required");
  const rkv_params& p = plan->params;
  const int n = (int)plan->layers.size();
  const int G = shape->n_q_heads / shape->n_kv_heads;
  // every layer is checked before anything is enqueued
  bool any = false;
  for (int l = 0; l < n; ++l) {
    const rkv_layer& ly = plan->layers[l];
    if (ly.rule_decode == RKV_FULL) continue;
    any = true;
    const int C = ly.budget_decode;
    if (position < C) return rkv::fail(RKV_ERR_SHAPE, "position must be >= the layer's capacity");
    const bool need_acc = ly.rule_decode == RKV_H2O;
    if (!state->k_cache[l] || !state->v_cache[l] || !state->pos[l] || (need_acc && (!state->acc || !state->acc[l])) ||
        !input->q[l] || !input->k[l] || !input->v[l])
      return rkv::fail(RKV_ERR_INVALID_ARG, "layer " + std::to_string(l) + ": null decode buffer");
    if ((size_t)(G + 1) * (C + 1) * sizeof(float) > 150 * 1024)
      return rkv::fail(RKV_ERR_UNSUPPORTED, "decode capacity too large for one workgroup's LDS");
  }
  if (any && G != 1 && G != 2 && G != 4 && G != 8)
    return rkv::fail(RKV_ERR_UNSUPPORTED, "decode needs n_q_heads / n_kv_heads in {1, 2, 4, 8}");
  for (int l0 = 0; l0 < n; l0 += rkv::kMaxLayersPerLaunch) {
    rkv::DecodeLaunch D;
    std::memset(&D, 0, sizeof(D));
    D.batch = shape->batch;
    D.n_q_heads = shape->n_q_heads;
    D.n_kv_heads = shape->n_kv_heads;
    D.group = G;
    D.position = position;
    D.n_sink = p.n_sink;
    D.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)shape->head_dim));
    int cnt = 0, max_cap = 0;
    for (int l = l0; l < std::min(n, l0 + rkv::kMaxLayersPerLaunch); ++l) {
      const rkv_layer& ly = plan->layers[l];
      if (ly.rule_decode == RKV_FULL) continue;
      const int C = ly.budget_decode;
      const bool need_acc = ly.rule_decode == RKV_H2O;
      rkv::DecodeLayer& d = D.layer[cnt++];
      d.k_cache = (uint16_t*)state->k_cache[l];
      d.v_cache = (uint16_t*)state->v_cache[l];
      d.pos = state->pos[l];
      d.acc = need_acc ? state->acc[l] : nullptr;
      d.q = (const uint16_t*)input->q[l];
      d.k = (const uint16_t*)input->k[l];
      d.v = (const uint16_t*)input->v[l];
      d.victim = input->victim_out ? input->victim_out[l] : nullptr;
      d.rule = ly.rule_decode;
      d.capacity = C;
      d.recent = (int32_t)(((int64_t)C * p.recent_num) / p.recent_den);
      max_cap = std::max(max_cap, C);
    }
    if (!cnt) continue;
    D.n_layers = cnt;
    int err = rkv::launch_decode(D, max_cap, stream);
    if (err) return rkv::fail(RKV_ERR_HIP, std::string("kernel launch failed: ") + hipGetErrorString((hipError_t)err));
  }
  return RKV_OK;
}

int rkv_decode_init_from_prefill(const rkv_plan* plan, const rkv_shape* shape, const rkv_prefill_io* prefill,
                                 const rkv_decode_state* state, void* stream) {
  rkv::clear_error();
  if (!plan || !prefill || !state) return rkv::fail(RKV_ERR_INVALID_ARG, "null plan, prefill io or state");
  int st = validate_shape(shape);
  if (st) return st;
  const int n = (int)plan->layers.size();
  const int L = shape->seq_len;
  const int64_t rows = (int64_t)shape->batch * shape->n_kv_heads;
  std::vector<rkv::CopyTask> tasks;
  for (int l = 0; l < n; ++l) {
    const rkv_layer& ly = plan->layers[l];
    if (ly.rule_decode == RKV_FULL) continue;
    const std::string at = "layer " + std::to_string(l) + ": ";
    const Layout lo = prefill_layout(ly, plan->params, L);
    const int C = ly.budget_decode;
    if (lo.n_keep != C)
      return rkv::fail(RKV_ERR_SHAPE, at + "decode capacity " + std::to_string(C) + " differs from the prefill retained count " +
                                          std::to_string(lo.n_keep));
    if (!prefill->k_out || !prefill->v_out || !prefill->idx_out || !prefill->k_out[l] || !prefill->v_out[l] ||
        !prefill->idx_out[l])
      return rkv::fail(RKV_ERR_INVALID_ARG, at + "null prefill output");
    if (!state->k_cache || !state->v_cache || !state->pos || !state->k_cache[l] || !state->v_cache[l] || !state->pos[l])
      return rkv::fail(RKV_ERR_INVALID_ARG, at + "null decode buffer");
    const int64_t kv_bytes = rows * C * rkv::kHeadDim * 2, pos_bytes = rows * C * 4;
    tasks.push_back({prefill->k_out[l], state->k_cache[l], kv_bytes});
    tasks.push_back({prefill->v_out[l], state->v_cache[l], kv_bytes});
    tasks.push_back({prefill->idx_out[l], state->pos[l], pos_bytes});
    if (ly.rule_decode == RKV_H2O) {
      if (!state->acc || !state->acc[l]) return rkv::fail(RKV_ERR_INVALID_ARG, at + "decode H2O needs acc");
      const bool scores = ly.rule_prefill != RKV_FULL && ly.rule_prefill != RKV_STREAMING;
      const float* src = prefill->acc_out ? prefill->acc_out[l] : nullptr;
      if (scores && !src)
        return rkv::fail(RKV_ERR_INVALID_ARG, at + "decode H2O is seeded from the prefill acc_out, which is null");
      tasks.push_back({src, state->acc[l], pos_bytes});   // null source: zero seed
    }
  }
  // drop copies onto themselves (a caller decoding in the prefill outputs)
  tasks.erase(std::remove_if(tasks.begin(), tasks.end(), [](const rkv::CopyTask& t) { return t.src == t.dst; }),
              tasks.end());
  for (size_t t0 = 0; t0 < tasks.size(); t0 += rkv::kMaxCopies) {
    rkv::CopyLaunch C;
    std::memset(&C, 0, sizeof(C));
    C.n_tasks = (int32_t)std::min<size_t>(rkv::kMaxCopies, tasks.size() - t0);
    for (int i = 0; i < C.n_tasks; ++i) C.task[i] = tasks[t0 + i];
    int err = rkv::launch_copies(C, stream);
    if (err) return rkv::fail(RKV_ERR_HIP, std::string("kernel launch failed: ") + hipGetErrorString((hipError_t)err));
  }
  return RKV_OK;
}

}  // extern "C"
