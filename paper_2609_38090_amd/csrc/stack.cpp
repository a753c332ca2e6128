// The GPU expert cache runtime behind mira_stack_* (paper sections IV-C, IV-D,
// IV-E, IV-F): HOT and STAGE slots of one pool shared by the layers of a
// model, demand fetches, the lookahead prefetch controller fed by a predictor
// head, per-expert telemetry and the bounded HOT rebalancer.
//
// All device work goes through the library's own calls (mira_moe_route,
// mira_moe_experts, mira_predict, mira_predict_mixture) and hipMemcpyAsync on
// the stack's copy stream; this file holds the host-side decisions and the
// stream/event plumbing.  Ordering rules:
//  - a copy into a slot waits (on the copy stream) for the event recorded
//    after the last layer whose experts read that slot, and nothing else;
//  - the compute stream waits for a slot's copy event once, before the first
//    layer that reads the slot after the copy;
//  - a layer's slot-table row is written by a small kernel on the compute
//    stream right before that layer's experts run.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <deque>
#include <numeric>
#include <vector>

#include "mira.h"
#include "mira_internal.h"

namespace {

using mira::set_error;

constexpr int kHistory = 8;            // past windows a telemetry record keeps
constexpr size_t kEventLogMax = 65536;  // logged events kept

enum Role { ROLE_HOT = 0, ROLE_STAGE = 1 };

struct Slot {
  int role = ROLE_STAGE;
  int layer = -1, expert = -1;  // content; -1 = free
  bool copy_pending = false;     // the compute stream has not yet waited for the copy
  hipEvent_t copied = nullptr;   // recorded on the copy stream after the copy into the slot
  int reader_layer = -1;         // last layer whose experts read the slot (its event in layer_done)
  uint64_t age = 0;              // clock of the copy that filled it
};

// Telemetry of one expert over the current window (section IV-D).
struct ExpertTel {
  int32_t routed = 0, hot = 0, stage = 0, cpu = 0;
  int64_t last_use = -1;
  std::deque<int32_t> history;  // routed volume of past windows, oldest first
};

struct LayerTel {
  std::vector<ExpertTel> e;
  int64_t tokens = 0, clock = 0;
  void close_window() {
    for (auto& x : e) {
      x.history.push_back(x.routed);
      if ((int)x.history.size() > kHistory) x.history.pop_front();
      x.routed = x.hot = x.stage = x.cpu = 0;
    }
    tokens = 0;
  }
};

struct Swap {
  int evict, promote;
};

// The rebalancer's plan for one layer (the order and rules of mira.h's
// mira_rebalance_plan).
std::vector<Swap> plan_swaps(const mira_stack_config& cfg, int n, const int32_t* routed,
                             const int32_t* cpu, const int64_t* last_use,
                             const std::vector<std::vector<int32_t>>& hist, const uint8_t* is_hot) {
  std::vector<int> victims, cands;
  for (int e = 0; e < n; ++e) {
    if (is_hot[e]) {
      victims.push_back(e);
      continue;
    }
    if (routed[e] <= 0) continue;
    const int need = cfg.rb_probation - 1;
    const auto& h = hist[e];
    bool probation = (int)h.size() < need;
    for (int i = 0; !probation && i < need; ++i)
      if (h[h.size() - 1 - i] == 0) probation = true;
    if (!probation) cands.push_back(e);
  }
  auto hsum = [&](int e) { return std::accumulate(hist[e].begin(), hist[e].end(), (int64_t)0); };
  std::sort(victims.begin(), victims.end(), [&](int a, int b) {
    if (routed[a] != routed[b]) return routed[a] < routed[b];
    if (last_use[a] != last_use[b]) return last_use[a] < last_use[b];
    const int64_t ha = hsum(a), hb = hsum(b);
    if (ha != hb) return ha < hb;
    return a < b;
  });
  auto score = [&](int e) { return (double)routed[e] + (double)cfg.rb_miss_weight * cpu[e]; };
  std::sort(cands.begin(), cands.end(), [&](int a, int b) {
    const double sa = score(a), sb = score(b);
    if (sa != sb) return sa > sb;
    return a < b;
  });
  std::vector<Swap> out;
  for (size_t i = 0; i < victims.size() && i < cands.size(); ++i) {
    if ((int)out.size() >= cfg.rb_max_swaps) break;
    if (score(cands[i]) < (double)routed[victims[i]] + cfg.rb_margin) break;
    out.push_back(Swap{victims[i], cands[i]});
  }
  return out;
}

}  // namespace

struct mira_stack {
  mira_stack_config cfg{};
  mira_shape shape{};
  int G = 0;        // experts per layer, routed then shared
  int n_slots = 0;
  int8_t* pool = nullptr;
  int32_t* tables = nullptr;  // device [L][G]
  hipStream_t compute = nullptr, copy = nullptr, side = nullptr;
  std::vector<Slot> slots;
  std::vector<std::vector<int>> hot;              // [L][G]: HOT slot or -1
  std::vector<std::vector<const void*>> host;     // [L][G]: CPU-store blob
  std::vector<std::vector<uint64_t>> host_bytes;  // [L][G]
  std::vector<LayerTel> tel;
  std::vector<std::vector<int>> predicted;        // [L]: the head's pick for that layer
  std::vector<hipEvent_t> layer_done;             // [L]: after the layer's experts
  hipEvent_t ev_counts = nullptr, ev_routed = nullptr, ev_scores = nullptr;
  hipEvent_t wall0 = nullptr, wall1 = nullptr;
  int32_t* counts_d = nullptr;  // device [G]
  int32_t* counts_h = nullptr;  // pinned [G]
  float* scores_d = nullptr;    // device [max_tokens][MIRA_MAX_EXPERTS]
  float* scores_h = nullptr;    // pinned, same size
  std::vector<std::pair<hipEvent_t, hipEvent_t>> copy_ev, stall_ev;  // timing pairs of the step
  std::vector<hipEvent_t> ev_pool;                                   // free timing events
  uint64_t clock = 0;
  bool in_step = false;
  mira_stack_stats cur{};
  std::deque<mira_stack_event> log;

  void note(int kind, int layer, int target, int expert, int slot) {
    if (log.size() >= kEventLogMax) log.pop_front();
    log.push_back(mira_stack_event{kind, layer, target, expert, slot, 0});
  }
  hipEvent_t timing_event() {
    if (!ev_pool.empty()) {
      hipEvent_t e = ev_pool.back();
      ev_pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};

namespace {

#define HIP_OR_FAIL(call)                                                                   \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return set_error(MIRA_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e_));       \
  } while (0)

#define MIRA_TRY(call)      \
  do {                      \
    int rc_ = (call);       \
    if (rc_) return rc_;    \
  } while (0)

int find_slot(const mira_stack* st, int layer, int expert, int role) {
  for (int i = 0; i < st->n_slots; ++i) {
    const Slot& s = st->slots[i];
    if (s.role == role && s.layer == layer && s.expert == expert) return i;
  }
  return -1;
}

// A STAGE slot for a copy made while layer cur is being run: a free slot,
// else the oldest slot of a passed layer; a demand copy may also take the
// oldest prefetch for a later layer.  Slots of layer cur are never taken.
int free_stage(const mira_stack* st, int cur, bool demand) {
  int best = -1;
  for (int pass = 0; pass < 2 && best < 0; ++pass) {
    if (pass == 1 && !demand) break;
    for (int i = 0; i < st->n_slots; ++i) {
      const Slot& s = st->slots[i];
      if (s.role != ROLE_STAGE) continue;
      const bool ok = pass == 0 ? (s.layer < 0 || s.layer < cur) : s.layer > cur;
      if (!ok) continue;
      if (pass == 0 && s.layer < 0) return i;  // a free slot first, lowest index
      if (best < 0 || s.age < st->slots[best].age) best = i;
    }
  }
  return best;
}

// Copy expert e of layer l from the CPU store into slot i (copy stream).
int copy_in(mira_stack* st, int i, int l, int e) {
  const void* src = st->host[l][e];
  const uint64_t bytes = st->host_bytes[l][e];
  if (!src)
    return set_error(MIRA_ERR_ARG, "expert %d of layer %d has no CPU-store blob (mira_stack_set_host)",
                     e, l);
  Slot& s = st->slots[i];
  if (s.reader_layer >= 0) HIP_OR_FAIL(hipStreamWaitEvent(st->copy, st->layer_done[s.reader_layer], 0));
  hipEvent_t t0 = st->timing_event(), t1 = st->timing_event();
  if (!t0 || !t1) return set_error(MIRA_ERR_HIP, "hipEventCreate failed");
  HIP_OR_FAIL(hipEventRecord(t0, st->copy));
  HIP_OR_FAIL(hipMemcpyAsync(st->pool + (size_t)i * st->cfg.slot_stride, src, bytes,
                             hipMemcpyHostToDevice, st->copy));
  HIP_OR_FAIL(hipEventRecord(t1, st->copy));
  HIP_OR_FAIL(hipEventRecord(s.copied, st->copy));
  st->copy_ev.emplace_back(t0, t1);
  st->cur.h2d_bytes += (int64_t)bytes;
  s.layer = l;
  s.expert = e;
  s.copy_pending = true;
  s.age = ++st->clock;
  return MIRA_OK;
}

// The compute stream waits for slot i's copy (once per copy).
int wait_copy(mira_stack* st, int i) {
  Slot& s = st->slots[i];
  if (!s.copy_pending) return MIRA_OK;
  hipEvent_t b = st->timing_event(), c = st->timing_event();
  if (!b || !c) return set_error(MIRA_ERR_HIP, "hipEventCreate failed");
  HIP_OR_FAIL(hipEventRecord(b, st->compute));
  HIP_OR_FAIL(hipStreamWaitEvent(st->compute, s.copied, 0));
  HIP_OR_FAIL(hipEventRecord(c, st->compute));
  st->stall_ev.emplace_back(b, c);
  s.copy_pending = false;
  return MIRA_OK;
}

// Stage expert e of layer l into a STAGE slot while layer cur runs; returns
// the slot, or -1 when a prefetch finds none (declined).
int stage(mira_stack* st, int cur, int l, int e, bool demand, int* slot_out) {
  const int i = free_stage(st, cur, demand);
  *slot_out = i;
  if (i < 0) {
    if (demand)
      return set_error(MIRA_ERR_UNSUPPORTED,
                       "no STAGE slot free for a demand copy of expert %d of layer %d: the stack "
                       "needs at least as many STAGE slots as non-HOT experts one layer selects",
                       e, l);
    return MIRA_OK;
  }
  const Slot& s = st->slots[i];
  if (demand && s.layer > cur) st->note(MIRA_EV_PREFETCH_DROPPED, cur, s.layer, s.expert, i);
  return copy_in(st, i, l, e);
}

int check_layer_args(const mira_stack* st, int layer, const mira_moe_args* a,
                     const mira_stack_head* h) {
  if (!a) return set_error(MIRA_ERR_ARG, "args is NULL");
  if (layer < 0 || layer >= st->cfg.n_layers) return set_error(MIRA_ERR_ARG, "layer %d out of range", layer);
  if (a->n_tokens < 1 || a->n_tokens > st->cfg.max_tokens)
    return set_error(MIRA_ERR_SHAPE, "n_tokens %d outside 1..max_tokens (%d)", a->n_tokens,
                     st->cfg.max_tokens);
  if (!st->in_step) return set_error(MIRA_ERR_ARG, "mira_stack_layer outside begin_step/end_step");
  if (h && (h->kind < MIRA_HEAD_NONE || h->kind > MIRA_HEAD_GIVEN))
    return set_error(MIRA_ERR_ARG, "bad head kind %d", h->kind);
  if (h && h->kind == MIRA_HEAD_GIVEN && h->n_given > 0 && !h->given)
    return set_error(MIRA_ERR_ARG, "head lists n_given experts but given is NULL");
  if (h && h->kind == MIRA_HEAD_MIXTURE && (!a->logits || !a->topk_idx || !h->mix || !h->mix_shape))
    return set_error(MIRA_ERR_ARG, "a MixtureHead needs the layer's logits and topk_idx outputs");
  if (h && h->kind == MIRA_HEAD_MLP && !h->mlp_shape)
    return set_error(MIRA_ERR_ARG, "an MLP head needs mlp_shape");
  return MIRA_OK;
}

// The head's pick for layer `tgt`: best stage_per_layer experts by the
// summed scores (ties to the lower index), or the given list.
int head_pick(mira_stack* st, const mira_stack_head* h, int n_groups, int n_out, std::vector<int>& want) {
  want.clear();
  if (h->kind == MIRA_HEAD_GIVEN) {
    for (int i = 0; i < h->n_given; ++i) {
      const int e = h->given[i];
      if (e < 0 || e >= st->G) return set_error(MIRA_ERR_ARG, "given expert %d out of range", e);
      if (std::find(want.begin(), want.end(), e) == want.end()) want.push_back(e);
    }
    return MIRA_OK;
  }
  HIP_OR_FAIL(hipEventSynchronize(st->ev_scores));
  std::vector<double> sum(n_out, 0.0);
  for (int g = 0; g < n_groups; ++g)
    for (int e = 0; e < n_out; ++e) sum[e] += st->scores_h[(size_t)g * n_out + e];
  std::vector<int> order(n_out);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return sum[a] > sum[b]; });
  const int m = std::min(st->cfg.stage_per_layer, n_out);
  want.assign(order.begin(), order.begin() + m);
  return MIRA_OK;
}

}  // namespace

namespace mira {
// The layer's slot-table row, by value, written on the stream (route.hip).
hipError_t launch_set_table(int32_t* table, const int32_t* row, int n, hipStream_t st);
}  // namespace mira

extern "C" {

int mira_rebalance_plan(const mira_stack_config* cfg, int32_t n_experts, const int32_t* routed,
                        const int32_t* cpu, const int64_t* last_use, const int32_t* history,
                        const int32_t* hist_len, const uint8_t* is_hot, int32_t max_swaps_out,
                        int32_t* evict, int32_t* promote, int32_t* n_swaps) {
  if (!cfg || !routed || !cpu || !last_use || !history || !hist_len || !is_hot || !evict || !promote ||
      !n_swaps)
    return set_error(MIRA_ERR_ARG, "NULL argument");
  if (n_experts < 1 || n_experts > MIRA_MAX_EXPERTS) return set_error(MIRA_ERR_SHAPE, "n_experts out of range");
  if (cfg->rb_probation < 1 || cfg->rb_max_swaps < 0) return set_error(MIRA_ERR_ARG, "bad rebalancer settings");
  std::vector<std::vector<int32_t>> hist(n_experts);
  for (int e = 0; e < n_experts; ++e) {
    if (hist_len[e] < 0 || hist_len[e] > kHistory) return set_error(MIRA_ERR_ARG, "hist_len out of range");
    hist[e].assign(history + (size_t)e * kHistory, history + (size_t)e * kHistory + hist_len[e]);
  }
  const auto sw = plan_swaps(*cfg, n_experts, routed, cpu, last_use, hist, is_hot);
  const int n = std::min<int>((int)sw.size(), max_swaps_out);
  for (int i = 0; i < n; ++i) {
    evict[i] = sw[i].evict;
    promote[i] = sw[i].promote;
  }
  *n_swaps = n;
  return mira::clear_error();
}

int mira_stack_create(const mira_stack_config* cfg, const mira_shape* s, void* slot_pool,
                      int32_t* slot_tables, hipStream_t compute, mira_stack** out) {
  if (!cfg || !s || !out) return set_error(MIRA_ERR_ARG, "NULL argument");
  *out = nullptr;
  if (cfg->n_layers < 1 || cfg->n_hot < 0 || cfg->n_stage < 0 || cfg->n_hot + cfg->n_stage < 1)
    return set_error(MIRA_ERR_SHAPE, "need n_layers >= 1 and at least one slot");
  if (cfg->max_tokens < 1) return set_error(MIRA_ERR_SHAPE, "max_tokens must be >= 1");
  if (cfg->vram_mode != MIRA_VRAM_LARGE && cfg->vram_mode != MIRA_VRAM_SMALL)
    return set_error(MIRA_ERR_ARG, "bad vram_mode");
  if (cfg->lookahead < 1 || cfg->stage_per_layer < 1)
    return set_error(MIRA_ERR_ARG, "lookahead and stage_per_layer must be >= 1");
  if (cfg->rb_interval < 0 || (cfg->rb_interval > 0 && (cfg->rb_probation < 1 || cfg->rb_max_swaps < 0)))
    return set_error(MIRA_ERR_ARG, "bad rebalancer settings");
  const bool i4 = s->flags & MIRA_FLAG_INT4;
  const size_t need = i4 ? mira_packed_expert_bytes_int4(s->hidden, s->ffn)
                         : mira_packed_expert_bytes(s->hidden, s->ffn);
  if (need == 0 || s->n_experts < 1 || s->n_shared < 0 || s->n_experts + s->n_shared > MIRA_MAX_EXPERTS)
    return set_error(MIRA_ERR_SHAPE, "bad layer shape");
  if (cfg->slot_stride % 256 || cfg->slot_stride < need)
    return set_error(MIRA_ERR_SHAPE, "slot_stride must be a multiple of 256 and >= %zu", need);
  if (!slot_pool || !slot_tables) return set_error(MIRA_ERR_ARG, "slot_pool and slot_tables are required");
  if ((uintptr_t)slot_pool % 256) return set_error(MIRA_ERR_ALIGN, "slot_pool must be 256-byte aligned");

  mira_stack* st = new (std::nothrow) mira_stack();
  if (!st) return set_error(MIRA_ERR_ARG, "out of host memory");
  st->cfg = *cfg;
  st->shape = *s;
  st->G = s->n_experts + s->n_shared;
  st->n_slots = cfg->n_hot + cfg->n_stage;
  st->pool = (int8_t*)slot_pool;
  st->tables = slot_tables;
  st->compute = compute;
  const int L = cfg->n_layers, G = st->G;
  st->slots.resize(st->n_slots);
  for (int i = 0; i < st->n_slots; ++i) st->slots[i].role = i < cfg->n_hot ? ROLE_HOT : ROLE_STAGE;
  st->hot.assign(L, std::vector<int>(G, -1));
  st->host.assign(L, std::vector<const void*>(G, nullptr));
  st->host_bytes.assign(L, std::vector<uint64_t>(G, 0));
  st->tel.resize(L);
  for (auto& t : st->tel) t.e.resize(G);
  st->predicted.assign(L, {});
  st->layer_done.assign(L, nullptr);

  auto bail = [&](hipError_t e, const char* what) {
    mira_stack_destroy(st);
    return set_error(MIRA_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
  };
  hipError_t e;
  // every stream keeps the default priority
  if ((e = hipStreamCreateWithFlags(&st->copy, hipStreamNonBlocking)) != hipSuccess) return bail(e, "hipStreamCreate");
  if ((e = hipStreamCreateWithFlags(&st->side, hipStreamNonBlocking)) != hipSuccess) return bail(e, "hipStreamCreate");
  for (auto& s2 : st->slots)
    if ((e = hipEventCreateWithFlags(&s2.copied, hipEventDisableTiming)) != hipSuccess) return bail(e, "hipEventCreate");
  for (auto& ev : st->layer_done)
    if ((e = hipEventCreateWithFlags(&ev, hipEventDisableTiming)) != hipSuccess) return bail(e, "hipEventCreate");
  for (hipEvent_t* ev : {&st->ev_counts, &st->ev_routed, &st->ev_scores})
    if ((e = hipEventCreateWithFlags(ev, hipEventDisableTiming)) != hipSuccess) return bail(e, "hipEventCreate");
  for (hipEvent_t* ev : {&st->wall0, &st->wall1})
    if ((e = hipEventCreate(ev)) != hipSuccess) return bail(e, "hipEventCreate");
  if ((e = hipMalloc((void**)&st->counts_d, sizeof(int32_t) * G)) != hipSuccess) return bail(e, "hipMalloc");
  if ((e = hipHostMalloc((void**)&st->counts_h, sizeof(int32_t) * G, hipHostMallocDefault)) != hipSuccess)
    return bail(e, "hipHostMalloc");
  const size_t sc = (size_t)cfg->max_tokens * MIRA_MAX_EXPERTS * sizeof(float);
  if ((e = hipMalloc((void**)&st->scores_d, sc)) != hipSuccess) return bail(e, "hipMalloc");
  if ((e = hipHostMalloc((void**)&st->scores_h, sc, hipHostMallocDefault)) != hipSuccess)
    return bail(e, "hipHostMalloc");
  // every table entry starts as "not resident"
  std::vector<int32_t> neg((size_t)L * G, -1);
  if ((e = hipMemcpyAsync(slot_tables, neg.data(), neg.size() * 4, hipMemcpyHostToDevice, compute)) !=
      hipSuccess)
    return bail(e, "hipMemcpyAsync");
  if ((e = hipStreamSynchronize(compute)) != hipSuccess) return bail(e, "hipStreamSynchronize");
  *out = st;
  return mira::clear_error();
}

int mira_stack_destroy(mira_stack* st) {
  if (!st) return mira::clear_error();
  // let queued work that uses the stack's buffers finish first; teardown
  // goes on whatever these calls return
  if (st->copy) (void)hipStreamSynchronize(st->copy);
  if (st->side) (void)hipStreamSynchronize(st->side);
  if (st->compute) (void)hipStreamSynchronize(st->compute);
  for (auto& s : st->slots)
    if (s.copied) (void)hipEventDestroy(s.copied);
  for (auto ev : st->layer_done)
    if (ev) (void)hipEventDestroy(ev);
  for (hipEvent_t ev : {st->ev_counts, st->ev_routed, st->ev_scores, st->wall0, st->wall1})
    if (ev) (void)hipEventDestroy(ev);
  for (auto& p : st->copy_ev) {
    (void)hipEventDestroy(p.first);
    (void)hipEventDestroy(p.second);
  }
  for (auto& p : st->stall_ev) {
    (void)hipEventDestroy(p.first);
    (void)hipEventDestroy(p.second);
  }
  for (auto ev : st->ev_pool) (void)hipEventDestroy(ev);
  if (st->counts_d) (void)hipFree(st->counts_d);
  if (st->counts_h) (void)hipHostFree(st->counts_h);
  if (st->scores_d) (void)hipFree(st->scores_d);
  if (st->scores_h) (void)hipHostFree(st->scores_h);
  if (st->copy) (void)hipStreamDestroy(st->copy);
  if (st->side) (void)hipStreamDestroy(st->side);
  delete st;
  return mira::clear_error();
}

int mira_stack_set_host(mira_stack* st, int32_t layer, int32_t expert, const void* pinned,
                        uint64_t bytes) {
  if (!st) return set_error(MIRA_ERR_ARG, "stack is NULL");
  if (layer < 0 || layer >= st->cfg.n_layers || expert < 0 || expert >= st->G)
    return set_error(MIRA_ERR_ARG, "layer or expert out of range");
  if (bytes > st->cfg.slot_stride) return set_error(MIRA_ERR_SHAPE, "blob larger than a slot");
  st->host[layer][expert] = pinned;
  st->host_bytes[layer][expert] = pinned ? bytes : 0;
  return mira::clear_error();
}

int mira_stack_set_hot(mira_stack* st, int32_t layer, int32_t expert, int32_t slot, int32_t copy) {
  if (!st) return set_error(MIRA_ERR_ARG, "stack is NULL");
  if (layer < 0 || layer >= st->cfg.n_layers || expert < 0 || expert >= st->G)
    return set_error(MIRA_ERR_ARG, "layer or expert out of range");
  // the HOT region is the first n_hot slots until rebalancing relabels slots
  if (slot < 0 || slot >= st->n_slots || st->slots[slot].role != ROLE_HOT)
    return set_error(MIRA_ERR_ARG, "slot %d is not a HOT slot", slot);
  Slot& s = st->slots[slot];
  if (s.layer >= 0 && s.expert >= 0 && st->hot[s.layer][s.expert] == slot) st->hot[s.layer][s.expert] = -1;
  if (st->hot[layer][expert] >= 0) st->slots[st->hot[layer][expert]].layer = -1;
  st->hot[layer][expert] = slot;
  if (copy) {
    MIRA_TRY(copy_in(st, slot, layer, expert));
  } else {
    s.layer = layer;
    s.expert = expert;
    s.copy_pending = false;
  }
  return mira::clear_error();
}

int mira_stack_begin_step(mira_stack* st) {
  if (!st) return set_error(MIRA_ERR_ARG, "stack is NULL");
  if (st->in_step) return set_error(MIRA_ERR_ARG, "a step is already open");
  HIP_OR_FAIL(hipEventRecord(st->wall0, st->compute));
  st->in_step = true;
  return mira::clear_error();
}

int mira_stack_layer(mira_stack* st, int32_t l, const mira_moe_args* a_in, const mira_stack_head* head) {
  if (!st) return set_error(MIRA_ERR_ARG, "stack is NULL");
  MIRA_TRY(check_layer_args(st, l, a_in, head));
  const int G = st->G, E = st->shape.n_experts, L = st->cfg.n_layers;
  mira_moe_args a = *a_in;
  a.slot_table = st->tables + (size_t)l * G;
  a.slot_pool = st->pool;
  a.n_slots = st->n_slots;
  a.slot_stride = st->cfg.slot_stride;
  int32_t* counts = a.expert_counts ? a.expert_counts : st->counts_d;
  a.expert_counts = counts;
  const int tgt = l + st->cfg.lookahead;
  const int kind = (head && tgt < L) ? head->kind : MIRA_HEAD_NONE;

  // 1. routing, and the head for layer l + lookahead beside the experts
  MIRA_TRY(mira_moe_route(&st->shape, &a, st->compute));
  int n_groups = 0, n_out = 0;
  if (kind == MIRA_HEAD_MLP || kind == MIRA_HEAD_MIXTURE) {
    HIP_OR_FAIL(hipEventRecord(st->ev_routed, st->compute));
    HIP_OR_FAIL(hipStreamWaitEvent(st->side, st->ev_routed, 0));
    if (kind == MIRA_HEAD_MLP) {
      const mira_pred_shape& p = *head->mlp_shape;
      n_groups = p.group > 0 ? a.n_tokens / p.group : 0;
      n_out = p.n_out;
      if (n_out < 1 || n_out > MIRA_MAX_EXPERTS) return set_error(MIRA_ERR_SHAPE, "head n_out out of range");
      MIRA_TRY(mira_predict(&p, a.x, a.n_tokens, head->w1, head->b1, head->w2, head->b2, st->scores_d,
                            head->workspace, head->workspace_bytes, st->side));
    } else {
      const mira_mixture_shape& p = *head->mix_shape;
      n_groups = p.group > 0 ? a.n_tokens / p.group : 0;
      n_out = p.n_out;
      if (n_out < 1 || n_out > MIRA_MAX_EXPERTS) return set_error(MIRA_ERR_SHAPE, "head n_out out of range");
      MIRA_TRY(mira_predict_mixture(&p, head->mix, a.x, a.logits, a.topk_idx, a.n_tokens, st->scores_d,
                                    nullptr, head->workspace, head->workspace_bytes, st->side));
    }
    HIP_OR_FAIL(hipMemcpyAsync(st->scores_h, st->scores_d, sizeof(float) * n_groups * n_out,
                               hipMemcpyDeviceToHost, st->side));
    HIP_OR_FAIL(hipEventRecord(st->ev_scores, st->side));
  }
  HIP_OR_FAIL(hipMemcpyAsync(st->counts_h, counts, sizeof(int32_t) * G, hipMemcpyDeviceToHost, st->compute));
  HIP_OR_FAIL(hipEventRecord(st->ev_counts, st->compute));
  HIP_OR_FAIL(hipEventSynchronize(st->ev_counts));
  std::vector<int32_t> cnt(st->counts_h, st->counts_h + G);

  // Coverage@m of the prediction made for this layer, if any
  if (!st->predicted[l].empty()) {
    int64_t tot = 0, hit = 0;
    for (int e = 0; e < E; ++e) tot += cnt[e];
    for (int e : st->predicted[l])
      if (e < E) hit += cnt[e];
    st->cur.cov_hits += hit;
    st->cur.cov_total += tot;
    st->predicted[l].clear();
  }

  // 2. serve every selected expert
  LayerTel& tel = st->tel[l];
  std::vector<int32_t> row(G, -1);
  std::vector<int> used;
  for (int e = 0; e < G; ++e) {
    if (cnt[e] <= 0) continue;
    int slot = st->hot[l][e];
    ExpertTel& t = tel.e[e];
    if (slot >= 0) {
      st->cur.hot_hits++;
      st->cur.hot_tokens += cnt[e];
      t.hot += cnt[e];
      st->note(MIRA_EV_HOT_HIT, l, l, e, slot);
    } else if ((slot = find_slot(st, l, e, ROLE_STAGE)) >= 0) {
      st->cur.stage_hits++;
      st->cur.stage_tokens += cnt[e];
      t.stage += cnt[e];
      st->note(MIRA_EV_STAGE_HIT, l, l, e, slot);
    } else {
      MIRA_TRY(stage(st, l, l, e, true, &slot));
      st->cur.misses++;
      st->cur.cpu_tokens += cnt[e];
      t.cpu += cnt[e];
      st->note(MIRA_EV_DEMAND, l, l, e, slot);
    }
    t.routed += cnt[e];
    t.last_use = tel.clock;
    MIRA_TRY(wait_copy(st, slot));
    row[e] = slot;
    used.push_back(slot);
  }
  tel.tokens += a.n_tokens;
  tel.clock += a.n_tokens;

  // 3. the layer's table row, then its experts
  HIP_OR_FAIL(mira::launch_set_table(st->tables + (size_t)l * G, row.data(), G, st->compute));
  MIRA_TRY(mira_moe_experts(&st->shape, &a, st->compute));
  HIP_OR_FAIL(hipEventRecord(st->layer_done[l], st->compute));
  for (int i : used) st->slots[i].reader_layer = l;
  if (st->cfg.vram_mode == MIRA_VRAM_SMALL)
    for (auto& s : st->slots)
      if (s.role == ROLE_STAGE && s.layer == l) s.layer = s.expert = -1;

  // 4. prefetch for layer l + lookahead
  if (kind != MIRA_HEAD_NONE) {
    std::vector<int> want;
    MIRA_TRY(head_pick(st, head, n_groups, n_out, want));
    st->predicted[tgt] = want;
    for (int e : want) {
      st->note(MIRA_EV_PREDICTED, l, tgt, e, -1);
      if (e >= G) continue;
      int slot = st->hot[tgt][e];
      if (slot < 0) slot = find_slot(st, tgt, e, ROLE_STAGE);
      if (slot >= 0) {
        st->cur.prefetch_cached++;
        st->note(MIRA_EV_PREFETCH_CACHED, l, tgt, e, slot);
        continue;
      }
      MIRA_TRY(stage(st, l + 1, tgt, e, false, &slot));
      if (slot < 0) {
        st->cur.prefetch_declined++;
        st->note(MIRA_EV_PREFETCH_DECLINED, l, tgt, e, -1);
      } else {
        st->cur.prefetches++;
        st->note(MIRA_EV_PREFETCH, l, tgt, e, slot);
      }
    }
  }

  // 5. HOT rebalancing (section IV-D)
  if (st->cfg.rb_interval > 0 && tel.tokens >= st->cfg.rb_interval) {
    std::vector<int32_t> routed(G), cpu(G);
    std::vector<int64_t> last(G);
    std::vector<std::vector<int32_t>> hist(G);
    std::vector<uint8_t> is_hot(G);
    for (int e = 0; e < G; ++e) {
      routed[e] = tel.e[e].routed;
      cpu[e] = tel.e[e].cpu;
      last[e] = tel.e[e].last_use;
      hist[e].assign(tel.e[e].history.begin(), tel.e[e].history.end());
      is_hot[e] = st->hot[l][e] >= 0;
    }
    for (const Swap& sw : plan_swaps(st->cfg, G, routed.data(), cpu.data(), last.data(), hist, is_hot.data())) {
      const int sv = st->hot[l][sw.evict];
      st->hot[l][sw.evict] = -1;
      st->note(MIRA_EV_EVICT, l, l, sw.evict, sv);
      const int sc = find_slot(st, l, sw.promote, ROLE_STAGE);
      if (sc >= 0) {
        // the staged copy becomes the HOT copy; the victim's slot joins STAGE
        st->slots[sc].role = ROLE_HOT;
        st->slots[sv].role = ROLE_STAGE;
        st->slots[sv].layer = st->slots[sv].expert = -1;
        st->slots[sv].copy_pending = false;
        st->hot[l][sw.promote] = sc;
        st->note(MIRA_EV_SWAP_RELABEL, l, l, sw.promote, sc);
      } else {
        MIRA_TRY(copy_in(st, sv, l, sw.promote));
        st->hot[l][sw.promote] = sv;
        st->cur.promote_copies++;
        st->note(MIRA_EV_SWAP_COPY, l, l, sw.promote, sv);
      }
      st->cur.swaps++;
    }
    tel.close_window();
  }
  return mira::clear_error();
}

int mira_stack_end_step(mira_stack* st, mira_stack_stats* stats) {
  if (!st) return set_error(MIRA_ERR_ARG, "stack is NULL");
  if (!st->in_step) return set_error(MIRA_ERR_ARG, "no step is open");
  st->in_step = false;
  HIP_OR_FAIL(hipEventRecord(st->wall1, st->compute));
  HIP_OR_FAIL(hipStreamSynchronize(st->copy));
  HIP_OR_FAIL(hipStreamSynchronize(st->side));
  HIP_OR_FAIL(hipEventSynchronize(st->wall1));
  float ms = 0.f;
  HIP_OR_FAIL(hipEventElapsedTime(&ms, st->wall0, st->wall1));
  st->cur.wall_ms += ms;
  for (auto* v : {&st->copy_ev, &st->stall_ev}) {
    double sum = 0.0;
    for (auto& p : *v) {
      float t = 0.f;
      if (hipEventElapsedTime(&t, p.first, p.second) == hipSuccess) sum += t;
      st->ev_pool.push_back(p.first);
      st->ev_pool.push_back(p.second);
    }
    (v == &st->copy_ev ? st->cur.copy_ms : st->cur.stall_ms) += sum;
    v->clear();
  }
  if (stats) {
    const mira_stack_stats& c = st->cur;
#define MIRA_ADD(f) stats->f += c.f
    MIRA_ADD(hot_hits); MIRA_ADD(stage_hits); MIRA_ADD(misses);
    MIRA_ADD(hot_tokens); MIRA_ADD(stage_tokens); MIRA_ADD(cpu_tokens);
    MIRA_ADD(prefetches); MIRA_ADD(prefetch_cached); MIRA_ADD(prefetch_declined);
    MIRA_ADD(swaps); MIRA_ADD(promote_copies); MIRA_ADD(h2d_bytes);
    MIRA_ADD(cov_hits); MIRA_ADD(cov_total);
    MIRA_ADD(copy_ms); MIRA_ADD(stall_ms); MIRA_ADD(wall_ms);
#undef MIRA_ADD
  }
  st->cur = mira_stack_stats{};
  return mira::clear_error();
}

int mira_stack_reset_stage(mira_stack* st) {
  if (!st) return set_error(MIRA_ERR_ARG, "stack is NULL");
  HIP_OR_FAIL(hipStreamSynchronize(st->copy));
  HIP_OR_FAIL(hipStreamSynchronize(st->compute));
  for (auto& s : st->slots)
    if (s.role == ROLE_STAGE) {
      s.layer = s.expert = -1;
      s.copy_pending = false;
    }
  for (auto& p : st->predicted) p.clear();
  return mira::clear_error();
}

int32_t mira_stack_find(const mira_stack* st, int32_t layer, int32_t expert, int32_t role) {
  if (!st || layer < 0 || layer >= st->cfg.n_layers || expert < 0 || expert >= st->G) return -1;
  if (role == ROLE_HOT) return st->hot[layer][expert];
  if (role == ROLE_STAGE) return find_slot(st, layer, expert, ROLE_STAGE);
  return -1;
}

int mira_stack_read_events(mira_stack* st, int32_t max_events, mira_stack_event* events,
                           int32_t* n_events) {
  if (!st || !n_events || (max_events > 0 && !events)) return set_error(MIRA_ERR_ARG, "NULL argument");
  int n = 0;
  while (n < max_events && !st->log.empty()) {
    events[n++] = st->log.front();
    st->log.pop_front();
  }
  *n_events = n;
  return mira::clear_error();
}

}  // extern "C"
