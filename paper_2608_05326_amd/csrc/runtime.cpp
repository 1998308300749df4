// Host runtime of the QEvict tiered decode-step library: configuration
// checks, workspace planning, per-layer protocol state, kernel launches and
// the synchronous inspection calls.  No device memory is ever allocated here.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/qevict.h"
#include "qv_layout.h"

namespace qv {
struct AttnArgs;
struct RetierArgs;
struct MigrateArgs;
struct PackArgs;
}  // namespace qv
#include "qv_device.h"

namespace qv {
hipError_t launch_attend(const AttnArgs& a, hipStream_t st);
hipError_t launch_merge(const AttnArgs& a, hipStream_t st);
hipError_t launch_retier(const RetierArgs& a, hipStream_t st);
hipError_t launch_manual_move(const RetierArgs& a, int seq, int window, int to_quant, hipStream_t st);
hipError_t launch_init_units(const Geometry& g, const UnitLayout& L, uint8_t* base, int n_units,
                             hipStream_t st);
hipError_t launch_gate_publish(uint64_t* seq, uint64_t value, int32_t* clear, hipStream_t st);
hipError_t attend_footprint(const Geometry& g, int* vgprs, size_t* lds);
hipError_t migrate_footprint(const Geometry& g, int* vgprs, size_t* lds);
hipError_t launch_gate_wait(const uint64_t* seq, uint64_t value, int32_t* fail, int64_t ticks,
                            hipStream_t st);
hipError_t launch_migrate(const MigrateArgs& a, int max_quant, int max_promote, hipStream_t st);
hipError_t launch_pack_tokens(const PackArgs& a, hipStream_t st);
hipError_t launch_key_norm_init(const KeyNormArgs& a, hipStream_t st);
hipError_t launch_score_pow(const ScorePowArgs& a, hipStream_t st);
hipError_t launch_prefill_scores(const ObsArgs& a, hipStream_t st);
hipError_t static_obs_scratch(void** ptr, const char** what);
}  // namespace qv

using namespace qv;
static_assert(kScorePnorm == QEVICT_SCORE_PNORM, "score mode numbering");
static_assert(kStaticObsScratchBytes == QEVICT_STATIC_SCRATCH_BYTES, "fixed scratch size");

namespace {

thread_local std::string g_last_error;

qevict_status fail(qevict_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

constexpr int64_t kHeaderBytes = 256;
// workspace header: the routing gate's published sequence number (uint64) and its
// failure word (int32)
constexpr int64_t kHdrGateSeq = 0;
constexpr int64_t kHdrGateFail = 8;
constexpr double kGateSeconds = 10.0;
constexpr int kNumTimed = 5;

int ceil_div(int a, int b) { return (a + b - 1) / b; }

struct LayerState {
  int T = 0;              // tokens held (all sequences)
  int routed_end = 0;     // windows below this index have been routed
  bool prefilled = false;
  bool period_start = false;    // a routing event (or prefill) since the last decode step
  int64_t last_bytes = 0;
};

struct TimedLaunch {
  int kernel;
  int units;   // layer routing events the launch serves (1 for other kernels)
  hipEvent_t start, stop;
};

struct RouteRequest {
  int layer;
  RetierUnit unit;
  int max_quant, max_promote;
};

}  // namespace

struct qevict_cache {
  qevict_config cfg;
  Geometry g;
  UnitLayout L;
  uint8_t* ws = nullptr;
  size_t ws_bytes = 0;
  hipStream_t stream = nullptr;
  void* static_scratch = nullptr;           // this device's fixed initial-score scratch
  // Asynchronous routing (QEVICT_FLAG_ASYNC_ROUTING): routing requests are queued
  // and launched on rstream in batches of route_batch layers, behind one wait
  // for the cache stream: a device-side gate (the cache stream publishes gate_seq
  // in the workspace header, the routing stream's first kernel waits for it) or a
  // queue-level wait on main_ev (queue_wait; see routing_fits_beside_attention).
  hipStream_t rstream = nullptr;
  bool queue_wait = false;
  hipEvent_t main_ev = nullptr;             // cache stream position of a queue-level wait
  uint64_t gate_seq = 0;                    // last number published for a batch
  int64_t gate_ticks = 0;                   // the gate's time limit in wall-clock ticks
  int64_t clock_khz = 0;                    // the wall clock's rate
  bool gate_release = true;                 // false only to test the time-out path
  std::vector<hipEvent_t> batch_ev;         // ring: end of a launched batch
  std::vector<char> batch_joined;           // the cache stream already waits for that batch
  int next_batch_ev = 0;
  int route_batch = 1;
  std::vector<RouteRequest> route_queue;    // requested, not launched yet
  std::vector<char> route_queued;           // per layer: in route_queue
  std::vector<int> route_ev_idx;            // per layer: batch_ev of launched, unjoined routing, or -1
  std::vector<LayerState> layers;
  bool poisoned = false;
  bool profiling = false;
  std::vector<TimedLaunch> pending;
  std::vector<hipEvent_t> free_events;
  double prof_ms[kNumTimed] = {0};
  int64_t prof_n[kNumTimed] = {0};
};

namespace {

qevict_status check_config(const qevict_config* c) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "config is NULL");
  if (c->abi_version != QEVICT_ABI_VERSION)
    return fail(QEVICT_ERR_UNSUPPORTED, "abi_version %d, library implements %d", c->abi_version,
                QEVICT_ABI_VERSION);
  if (c->batch < 1 || c->num_layers < 1 || c->num_q_heads < 1 || c->num_kv_heads < 1)
    return fail(QEVICT_ERR_INVALID_ARG, "batch, layers and head counts must be positive");
  if (c->num_q_heads % c->num_kv_heads != 0)
    return fail(QEVICT_ERR_INVALID_ARG, "num_q_heads %% num_kv_heads != 0");
  if (c->num_q_heads / c->num_kv_heads > kMaxGqa || c->num_q_heads > 64)
    return fail(QEVICT_ERR_UNSUPPORTED, "at most 16 query heads per KV head and 64 query heads");
  if (c->head_dim != kHeadDim) return fail(QEVICT_ERR_UNSUPPORTED, "head_dim must be 128");
  if (c->window_tokens != 8 && c->window_tokens != 32 && c->window_tokens != 64)
    return fail(QEVICT_ERR_UNSUPPORTED, "window_tokens must be 8, 32 or 64");
  if (c->window_tokens == 8) {
    if (c->group_size != 32)
      return fail(QEVICT_ERR_UNSUPPORTED, "8-token windows take value groups of 32 channels (group_size 32)");
    if (c->rope_base > 0.f)
      return fail(QEVICT_ERR_UNSUPPORTED, "the RoPE-aware tier needs windows of 32 or 64 tokens");
  } else if (c->group_size != c->window_tokens) {
    return fail(QEVICT_ERR_UNSUPPORTED, "group_size must equal window_tokens (32 or 64)");
  }
  if (c->quant_bits != 4 && c->quant_bits != 2 && c->quant_bits != QEVICT_BITS_MIXED_4_2)
    return fail(QEVICT_ERR_UNSUPPORTED, "quant_bits must be 4, 2 or 42");
  if (c->sink_tokens < 0 || c->recent_tokens < 0 || c->capacity_full < 0 || c->capacity_quant < 0)
    return fail(QEVICT_ERR_INVALID_ARG, "negative sink, recent or capacity");
  if (c->max_context <= c->sink_tokens)
    return fail(QEVICT_ERR_INVALID_ARG, "max_context must exceed sink_tokens");
  if (ceil_div(c->sink_tokens, c->window_tokens) > kMaxSinkWindows)
    return fail(QEVICT_ERR_UNSUPPORTED, "sink_tokens must span at most %d windows", kMaxSinkWindows);
  if (c->retier_interval < 1) return fail(QEVICT_ERR_INVALID_ARG, "retier_interval must be >= 1");
  if (c->out_dtype != QEVICT_OUT_F32 && c->out_dtype != QEVICT_OUT_BF16)
    return fail(QEVICT_ERR_INVALID_ARG, "out_dtype");
  if (c->flags & ~(QEVICT_FLAG_NO_PROMOTION | QEVICT_FLAG_DEBUG_MASSES | QEVICT_FLAG_ASYNC_ROUTING |
                   QEVICT_FLAG_ROUTING_QUEUE_WAIT | QEVICT_FLAG_ROUTING_DEVICE_WAIT))
    return fail(QEVICT_ERR_INVALID_ARG, "unknown flags 0x%x", c->flags);
  const uint32_t order_flags = c->flags & (QEVICT_FLAG_ROUTING_QUEUE_WAIT | QEVICT_FLAG_ROUTING_DEVICE_WAIT);
  if (order_flags && !(c->flags & QEVICT_FLAG_ASYNC_ROUTING))
    return fail(QEVICT_ERR_INVALID_ARG, "routing order flags need QEVICT_FLAG_ASYNC_ROUTING");
  if (order_flags == (QEVICT_FLAG_ROUTING_QUEUE_WAIT | QEVICT_FLAG_ROUTING_DEVICE_WAIT))
    return fail(QEVICT_ERR_INVALID_ARG, "at most one routing order flag");
  if (!(c->softmax_scale >= 0.f) || !std::isfinite(c->softmax_scale))
    return fail(QEVICT_ERR_INVALID_ARG, "softmax_scale");
  if (c->score_mode != QEVICT_SCORE_CUMULATIVE && c->score_mode != QEVICT_SCORE_DECAY &&
      c->score_mode != QEVICT_SCORE_KEY_NORM && c->score_mode != QEVICT_SCORE_PNORM)
    return fail(QEVICT_ERR_INVALID_ARG, "score_mode");
  if (!(c->rope_base >= 0.f) || !std::isfinite(c->rope_base))
    return fail(QEVICT_ERR_INVALID_ARG, "rope_base must be finite and >= 0");
  if (c->score_mode == QEVICT_SCORE_PNORM && !(c->score_p >= 1.f && c->score_p <= 16.f))
    return fail(QEVICT_ERR_INVALID_ARG, "score_p must be in [1, 16]");
  if (c->score_mode == QEVICT_SCORE_DECAY && !(c->score_decay > 0.f && c->score_decay <= 1.f))
    return fail(QEVICT_ERR_INVALID_ARG, "score_decay must be in (0, 1]");
  if (c->num_splits < 0 || c->num_splits > 256)
    return fail(QEVICT_ERR_INVALID_ARG, "num_splits must be in [0, 256]");
  if (c->num_splits * c->num_q_heads > 4096)
    return fail(QEVICT_ERR_UNSUPPORTED, "num_splits x num_q_heads must be <= 4096");
  const int W = c->window_tokens;
  const int nr = ceil_div(c->recent_tokens, W) + ceil_div(c->retier_interval, W) + 2;
  if (c->capacity_full + c->capacity_quant + nr > kMaxCand)
    return fail(QEVICT_ERR_UNSUPPORTED, "K_f + K_q + ring windows must be <= %d", kMaxCand);
  if (c->capacity_full + c->capacity_quant < 1)
    return fail(QEVICT_ERR_INVALID_ARG, "K_f + K_q must be >= 1");
  return QEVICT_OK;
}

void plan(const qevict_config* c, Geometry* g, UnitLayout* L) {
  memset(g, 0, sizeof *g);
  memset(L, 0, sizeof *L);
  g->B = c->batch;
  g->H_q = c->num_q_heads;
  g->H_kv = c->num_kv_heads;
  g->gqa = c->num_q_heads / c->num_kv_heads;
  g->d = c->head_dim;
  g->W = c->window_tokens;
  g->G = c->group_size;
  g->bits_cfg = c->quant_bits;
  g->qbits_max = c->quant_bits == 2 ? 2 : 4;
  g->K_f = c->capacity_full;
  g->K_q = c->capacity_quant;
  g->n_qslots = c->capacity_quant + c->capacity_full;
  {
    // the re-rank kernel keeps both owner tables (n_fslots + n_qslots entries)
    // in 2 * kMaxCand LDS words and scans each over at most kMaxCand entries
    int spare = kSpareFull;
    spare = std::min(spare, 2 * kMaxCand - 2 * g->K_f - g->K_q);
    spare = std::min(spare, kMaxCand - g->K_f);
    g->n_fslots = g->K_f + std::max(spare, 0);
  }
  g->NR = ceil_div(c->recent_tokens, g->W) + ceil_div(c->retier_interval, g->W) + 2;
  g->NS = ceil_div(c->sink_tokens, g->W);
  g->sink = c->sink_tokens;
  g->recent = c->recent_tokens;
  g->nwc = ceil_div(c->max_context - c->sink_tokens, g->W);
  g->max_fq = g->K_f + g->K_q;
  g->max_items = g->max_fq + g->NR + g->NS;
  int ns = c->num_splits;
  if (ns == 0) {
    // about two workgroups per compute unit over the whole grid
    ns = ceil_div(512, g->B * g->H_kv);
    ns = ns < 1 ? 1 : (ns > 64 ? 64 : ns);
    int per_split = ceil_div(g->max_items, ns);
    if (per_split < 2) ns = ceil_div(g->max_items, 2);
    if (ns * g->H_q > 4096) ns = 4096 / g->H_q;   // split statistics one merge thread folds
  }
  g->n_split = ns;
  g->out_bf16 = c->out_dtype == QEVICT_OUT_BF16;
  g->flags = c->flags;
  g->score_mode = c->score_mode;
  const float scale = c->softmax_scale > 0.f ? c->softmax_scale : 1.0f / std::sqrt((float)g->d);
  g->scale_log2 = scale * 1.4426950408889634f;
  g->fhead_bytes = (int64_t)g->W * g->d * 4;
  g->fslot_bytes = g->fhead_bytes * g->H_kv;
  g->qcodes_bytes = (int64_t)g->W * g->d * g->qbits_max / 8;
  g->qrec_bytes = 2 * g->qcodes_bytes + 4 * g->d + (int64_t)g->W * (g->d / g->G) * 4;
  g->qslot_bytes = g->qrec_bytes * g->H_kv;
  // split-balancing weights (per 32 tokens): a bf16 window moves twice the bytes
  // of an int4 one, which carries the code expansion instead; measured per-wave
  // times are close, so the weights are nearly equal.  An 8-token window costs
  // the same whatever its tier: its fixed per-window work outweighs its bytes.
  g->cost_bf16 = g->W == 8 ? 4 : 16 * (g->W / 32);
  g->cost_q4 = g->W == 8 ? 4 : 16 * (g->W / 32);
  g->cost_q2 = g->W == 8 ? 4 : 14 * (g->W / 32);
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    int64_t o = off;
    off = align256(off + bytes);
    return o;
  };
  L->fpool = take((int64_t)g->n_fslots * g->fslot_bytes);
  L->ring = take((int64_t)g->NR * g->fslot_bytes);
  L->sinkp = take((int64_t)g->NS * g->fslot_bytes);   // directly after the ring (zeroed together)
  L->qpool = take((int64_t)g->n_qslots * g->qslot_bytes);
  L->tier = take(g->nwc);
  L->ledger = take(g->nwc);
  L->bits = take(g->nwc);
  L->fslot = take(4LL * g->nwc);
  L->qslot = take(4LL * g->nwc);
  L->score = take(4LL * g->nwc);
  L->fowner = take(4LL * (g->n_fslots + 1));
  L->qowner = take(4LL * (g->n_qslots + 1));
  L->item_win = take(4LL * (g->max_fq + 1));
  L->item_ref = take(4LL * (g->max_fq + 1));
  L->item_cost = take(4LL * (g->max_fq + 1));
  L->item_aux = take(4LL * (g->max_fq + 1));
  L->item_score = take(4LL * (g->max_items + 1));
  L->qlist = take(4LL * kQEntry * (g->max_fq + 1));
  L->plist = take(4LL * kQEntry * (g->max_fq + 1));
  L->counts = take(4LL * CNT_N);
  L->stats = take(4LL * ST_N);
  L->partial = take(4LL * g->H_q * g->n_split * g->d);
  L->pml = take(8LL * g->H_q * g->n_split);
  L->mref = take(8LL * g->H_q * g->max_items);
  L->dbg_mass = take((c->flags & QEVICT_FLAG_DEBUG_MASSES) ? 4LL * g->H_q * (g->nwc + 1) : 0);
  L->plan = take(4LL * kPlanRec * 4 * g->n_split * kPlanSlots);
  L->pnorm = take(c->score_mode == QEVICT_SCORE_PNORM ? 8LL * g->nwc : 0);
  L->unit_bytes = align256(off);
}

bool ring_and_sink_adjacent(const UnitLayout& L, const Geometry& g) {
  return L.sinkp == align256(L.ring + (int64_t)g.NR * g.fslot_bytes);
}

qevict_status hip_fail(hipError_t e, const char* what) {
  return fail(QEVICT_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Key-norm and p-norm modes: prompt window scores are computed into a staging
// area after the units ([B][n_w] fp32), then routed like caller-supplied
// initial scores.
int64_t score_staging_bytes(const qevict_config* cfg, const Geometry& g) {
  const bool used = cfg->score_mode == QEVICT_SCORE_KEY_NORM || cfg->score_mode == QEVICT_SCORE_PNORM;
  return used ? align256(4LL * g.B * g.nwc) : 0;
}

// RoPE table after the staging area: (cos, sin) of p * base^(-2i/d), float32,
// [max_context][d / 2]
int64_t rope_table_bytes(const qevict_config* cfg) {
  return cfg->rope_base > 0.f ? align256(8LL * cfg->max_context * (cfg->head_dim / 2)) : 0;
}

std::vector<float> rope_table(const qevict_config* cfg) {
  const int half = cfg->head_dim / 2;
  std::vector<double> inv(half);
  for (int i = 0; i < half; ++i) inv[i] = std::pow((double)cfg->rope_base, -2.0 * i / cfg->head_dim);
  std::vector<float> t(2LL * cfg->max_context * half);
  for (int64_t p = 0; p < cfg->max_context; ++p)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)p * inv[i];
      t[2 * (p * half + i)] = (float)std::cos(ang);
      t[2 * (p * half + i) + 1] = (float)std::sin(ang);
    }
  return t;
}

uint8_t* unit_base(qevict_cache* c, int layer, int seq) {
  return c->ws + kHeaderBytes + ((int64_t)layer * c->g.B + seq) * c->L.unit_bytes;
}

// ---- kernel timing ----
hipEvent_t take_event(qevict_cache* c) {
  if (!c->free_events.empty()) {
    hipEvent_t e = c->free_events.back();
    c->free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void fold_pending(qevict_cache* c) {
  if (c->pending.empty()) return;
  for (auto& t : c->pending) (void)hipEventSynchronize(t.stop);   // launches may sit on two streams
  for (auto& t : c->pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.start, t.stop) == hipSuccess) {
      c->prof_ms[t.kernel] += ms;
      c->prof_n[t.kernel] += t.units;
    }
    c->free_events.push_back(t.start);
    c->free_events.push_back(t.stop);
  }
  c->pending.clear();
}

template <typename F>
hipError_t timed(qevict_cache* c, int kernel, hipStream_t st, F&& launch, int units = 1) {
  if (!c->profiling) return launch();
  if (c->pending.size() > 2048) fold_pending(c);
  hipEvent_t a = take_event(c), b = take_event(c);
  if (!a || !b) return launch();
  (void)hipEventRecord(a, st);
  hipError_t e = launch();
  (void)hipEventRecord(b, st);
  c->pending.push_back({kernel, units, a, b});
  return e;
}

// Whether a migration workgroup fits on a compute unit beside the two attention
// workgroups it holds during a decode step (both kernels run one wave per SIMD):
// registers of two attention waves and one migration wave per SIMD, LDS of the
// three workgroups.  Routing ordered by the device-side gate then proceeds beside
// attention.  Where it does not fit it waits for compute units that attention
// leaves free, and the queue-level wait, whose stall of the cache stream (about
// 12 us a batch) gives it that room, was measured faster: 128K context with
// 64-token windows (256-register attention), the RoPE-aware tier (256), GQA 8
// (217 plus a 79-register migration wave), 8-token windows (222 plus 96) with 16
// layer caches.
hipError_t routing_fits_beside_attention(const Geometry& g, bool* fits) {
  int av = 0, mv = 0;
  size_t al = 0, ml = 0;
  hipError_t e = attend_footprint(g, &av, &al);
  if (e == hipSuccess) e = migrate_footprint(g, &mv, &ml);
  if (e != hipSuccess) return e;
  auto granule = [](int v) { return (v + 7) / 8 * 8; };   // VGPR allocation granule
  *fits = 2 * granule(av) + granule(mv) <= 512 && 2 * al + ml <= 160 * 1024;
  return hipSuccess;
}

// Asynchronous routing: launch the queued routing requests on the routing
// stream, after everything enqueued on the cache stream so far.
hipError_t flush_routing(qevict_cache* c) {
  if (c->route_queue.empty()) return hipSuccess;
  hipStream_t rs = c->rstream;
  uint64_t* gate = (uint64_t*)(c->ws + kHdrGateSeq);
  int32_t* gate_fail = (int32_t*)(c->ws + kHdrGateFail);
  hipError_t e = hipSuccess;
  // A queue-level wait (a barrier packet on the routing stream waiting for the
  // cache stream's event) stalls the cache stream's own dispatches by about 12 us
  // a batch; the device-side gate does not.  The stall is what gives routing room
  // where its kernels do not fit beside attention (queue_wait, chosen at cache
  // creation by routing_fits_beside_attention or forced by a flag).
  if (c->queue_wait) {
    e = hipEventRecord(c->main_ev, c->stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(rs, c->main_ev, 0);
  } else {
    const uint64_t seq = ++c->gate_seq;
    if (c->gate_release) e = launch_gate_publish(gate, seq, nullptr, c->stream);
    if (e == hipSuccess) e = launch_gate_wait(gate, seq, gate_fail, c->gate_ticks, rs);
  }
  // one re-rank launch and one migration launch for the queued layers (distinct
  // layers: a layer is queued at most once)
  const int n = (int)c->route_queue.size();
  if (n > kRouteBatch) return hipErrorInvalidValue;   // (batches are flushed at route_batch <= kRouteBatch)
  RetierArgs ra{c->g, c->L, 0, nullptr, 0, n, {}, gate_fail};
  MigrateArgs ma{c->g, c->L, n, {}, nullptr, nullptr, 0, gate_fail};
  int mq = 0, mp = 0;
  for (int i = 0; i < n; ++i) {
    const RouteRequest& r = c->route_queue[i];
    ra.unit[i] = r.unit;
    ma.base[i] = r.unit.base;
    mq = std::max(mq, r.max_quant);
    mp = std::max(mp, r.max_promote);
  }
  if (e == hipSuccess) e = timed(c, 2, rs, [&] { return launch_retier(ra, rs); }, n);
  if (e == hipSuccess) e = timed(c, 3, rs, [&] { return launch_migrate(ma, mq, mp, rs); }, n);
  const int slot = c->next_batch_ev;
  c->next_batch_ev = (slot + 1) % (int)c->batch_ev.size();
  if (e == hipSuccess) e = hipEventRecord(c->batch_ev[slot], rs);
  c->batch_joined[slot] = 0;
  for (const RouteRequest& r : c->route_queue) {
    c->route_queued[r.layer] = 0;
    c->route_ev_idx[r.layer] = slot;
  }
  c->route_queue.clear();
  return e;
}

// Order the cache stream after the routing work of a layer (launching it first
// if it is still queued).  A finished batch needs no device-side wait.  An
// event of the ring may have been recorded again by a later batch; waiting on
// it then waits for more routing work than needed, never less.
hipError_t join_layer(qevict_cache* c, int layer) {
  if (!c->rstream) return hipSuccess;
  hipError_t e = hipSuccess;
  if (c->route_queued[layer] && (e = flush_routing(c)) != hipSuccess) return e;
  const int idx = c->route_ev_idx[layer];
  if (idx < 0) return hipSuccess;
  if (!c->batch_joined[idx]) {
    e = hipEventQuery(c->batch_ev[idx]);
    if (e == hipErrorNotReady) {
      e = hipStreamWaitEvent(c->stream, c->batch_ev[idx], 0);
      if (e == hipSuccess) c->batch_joined[idx] = 1;   // covers the batch's other layers too
    }
  }
  if (e == hipSuccess) c->route_ev_idx[layer] = -1;
  return e;
}

// Validates the handle and the layer; every later use of the layer on the
// cache stream is ordered after its pending routing work.
qevict_status check_handle(qevict_cache* c, int layer) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "cache is NULL");
  if (c->poisoned) return fail(QEVICT_ERR_BAD_STATE, "cache is in an error state; destroy it");
  if (layer < 0 || layer >= c->cfg.num_layers)
    return fail(QEVICT_ERR_INVALID_ARG, "layer %d out of range", layer);
  if (hipError_t e = join_layer(c, layer)) return hip_fail(e, "joining the routing stream");
  return QEVICT_OK;
}

qevict_status device_errors(qevict_cache* c, int layer) {
  int32_t cnt[CNT_N];
  for (int b = 0; b < c->g.B; ++b) {
    hipError_t e = hipMemcpyAsync(cnt, unit_base(c, layer, b) + c->L.counts, sizeof cnt,
                                  hipMemcpyDeviceToHost, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return hip_fail(e, "reading device error word");
    if (cnt[CNT_ERROR]) {
      c->poisoned = true;
      const int f = cnt[CNT_ERROR];
      if (f & ERR_NONFINITE) return fail(QEVICT_ERR_NONFINITE, "non-finite window score (seq %d)", b);
      if (f & ERR_RANGE) return fail(QEVICT_ERR_NONFINITE, "quantizer input outside fp16 range (seq %d)", b);
      if (f & ERR_GATE)
        return fail(QEVICT_ERR_BAD_STATE, "routing skipped: the routing stream waited more than %.0f s for "
                    "the cache stream (seq %d)", kGateSeconds, b);
      return fail(QEVICT_ERR_BAD_STATE, "device error flags 0x%x (seq %d)", f, b);
    }
  }
  return QEVICT_OK;
}

void fill_common(qevict_cache* c, int layer, Geometry* g, UnitLayout* L, uint8_t** base) {
  *g = c->g;
  *L = c->L;
  *base = unit_base(c, layer, 0);
}

int n_started(const Geometry& g, int T) { return T <= g.sink ? 0 : ceil_div(T - g.sink, g.W); }
// Split plans the re-rank kernel prepares for the decode steps up to the next
// routing event (sequence lengths T_next .. T_next + R - 1, windows below routed_end
// routed): consecutive steps with the same number of recent-region + sink windows
// share a plan slot; steps past the slots, past max_context or with more unrouted
// windows than the ring holds get none (the attention kernel then splits the list
// itself).
void plan_next(const Geometry& g, int max_context, int T_next, int R, int routed_end, RetierUnit* ra) {
  for (int j = 0; j < kPlanSlots; ++j) {
    ra->plan_t0[j] = -1;
    ra->plan_t1[j] = -2;
    ra->plan_extra[j] = 0;
  }
  int ns = 0;
  for (int k = 0; k < R; ++k) {
    const int T = T_next + k;
    const int n_ring = n_started(g, T) - routed_end;
    if (T > max_context || n_ring < 0 || n_ring > g.NR) break;
    const int extra = n_ring + g.NS;
    if (ns > 0 && extra == ra->plan_extra[ns - 1]) {
      ra->plan_t1[ns - 1] = T;
      continue;
    }
    if (ns == kPlanSlots) break;
    ra->plan_t0[ns] = ra->plan_t1[ns] = T;
    ra->plan_extra[ns] = extra;
    ++ns;
  }
}
int aged_end(const Geometry& g, int T) {
  int n = T - g.recent - g.sink;
  return n <= 0 ? 0 : n / g.W;
}

// double -> fp16 bits, round to nearest even (finite, in range)
uint16_t host_rne_fp16(double x) {
  uint16_t sign = std::signbit(x) ? 0x8000 : 0;
  double a = std::fabs(x);
  if (a == 0.0) return sign;
  int e;
  std::frexp(a, &e);              // a = m 2^e, m in [0.5, 1)
  int q = e - 11;                  // unit in the last place for 11 significant bits
  if (q < -24) q = -24;            // subnormal spacing
  double y = std::nearbyint(std::ldexp(a, -q));   // default rounding: ties to even
  double r = std::ldexp(y, q);
  if (r > 65504.0) return (uint16_t)(sign | 0x7C00);
  _Float16 h = (_Float16)(float)r;   // exact: r is an fp16 value
  uint16_t bits;
  memcpy(&bits, &h, 2);
  return (uint16_t)(bits | sign);
}

double host_fp16_to_double(uint16_t h) {
  _Float16 v;
  memcpy(&v, &h, 2);
  return (double)(float)v;
}

}  // namespace

extern "C" {

const char* qevict_status_string(qevict_status s) {
  switch (s) {
    case QEVICT_OK: return "ok";
    case QEVICT_ERR_INVALID_ARG: return "invalid argument";
    case QEVICT_ERR_UNSUPPORTED: return "unsupported";
    case QEVICT_ERR_WORKSPACE: return "workspace too small or misaligned";
    case QEVICT_ERR_BAD_STATE: return "bad state";
    case QEVICT_ERR_NONFINITE: return "non-finite value";
    case QEVICT_ERR_CAPACITY: return "capacity exceeded";
    case QEVICT_ERR_DEVICE: return "device error";
    default: return "unknown status";
  }
}

const char* qevict_last_error(void) { return g_last_error.c_str(); }

qevict_status qevict_capacities_for_budget(const qevict_config* cfg, int64_t budget_bytes,
                                           int32_t q_permille, int32_t* k_full, int32_t* k_quant) {
  if (!cfg || !k_full || !k_quant) return fail(QEVICT_ERR_INVALID_ARG, "null pointer");
  qevict_config c = *cfg;
  c.capacity_full = 1;   // capacities are the output: validate the rest
  c.capacity_quant = 0;
  qevict_status s = check_config(&c);
  if (s) return s;
  if (q_permille < 0 || q_permille > 1000) return fail(QEVICT_ERR_INVALID_ARG, "q_permille");
  const int64_t Hkv = c.num_kv_heads, d = c.head_dim, W = c.window_tokens, G = c.group_size;
  const int64_t bits = c.quant_bits == 2 ? 2 : 4;
  const int64_t protect = 4 * Hkv * d * ((int64_t)c.sink_tokens + c.recent_tokens);
  if (budget_bytes < protect)
    return fail(QEVICT_ERR_INVALID_ARG, "budget %lld below the protected regions (%lld bytes)",
                (long long)budget_bytes, (long long)protect);
  const int64_t hist = budget_bytes - protect;
  const int64_t m_f = 4 * Hkv * W * d + 8;
  const int64_t m_q = 2 * Hkv * W * d * bits / 8 + 4 * Hkv * d + 4 * Hkv * W * (d / G) + 10;
  // exact: floor(((1000 - q) / 1000) * hist / m_f); hist < 2^48 keeps the products in range
  if (hist >= ((int64_t)1 << 48)) return fail(QEVICT_ERR_INVALID_ARG, "budget too large");
  const int64_t kf = (1000 - q_permille) * hist / (1000 * m_f);
  const int64_t kq = q_permille * hist / (1000 * m_q);
  if (kf > INT32_MAX || kq > INT32_MAX) return fail(QEVICT_ERR_INVALID_ARG, "budget too large");
  *k_full = (int32_t)kf;
  *k_quant = (int32_t)kq;
  return QEVICT_OK;
}

qevict_status qevict_workspace_size(const qevict_config* cfg, size_t* bytes) {
  qevict_status s = check_config(cfg);
  if (s) return s;
  if (!bytes) return fail(QEVICT_ERR_INVALID_ARG, "bytes is NULL");
  Geometry g;
  UnitLayout L;
  plan(cfg, &g, &L);
  *bytes = (size_t)(kHeaderBytes + (int64_t)cfg->num_layers * cfg->batch * L.unit_bytes +
                    score_staging_bytes(cfg, g) + rope_table_bytes(cfg));
  return QEVICT_OK;
}

qevict_status qevict_cache_init(const qevict_config* cfg, void* workspace, size_t bytes,
                                void* hip_stream, qevict_cache** out) {
  qevict_status s = check_config(cfg);
  if (s) return s;
  if (!out) return fail(QEVICT_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  size_t need = 0;
  qevict_workspace_size(cfg, &need);
  if (!workspace || ((uintptr_t)workspace & 255))
    return fail(QEVICT_ERR_WORKSPACE, "workspace must be a 256-byte aligned device pointer");
  if (bytes < need) return fail(QEVICT_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, need);
  qevict_cache* c = new qevict_cache();
  c->cfg = *cfg;
  plan(cfg, &c->g, &c->L);
  if (!ring_and_sink_adjacent(c->L, c->g)) {
    delete c;
    return fail(QEVICT_ERR_UNSUPPORTED, "internal layout");
  }
  c->ws = (uint8_t*)workspace;
  c->ws_bytes = bytes;
  c->stream = (hipStream_t)hip_stream;
  c->layers.resize(cfg->num_layers);
  hipError_t e = hipSuccess;
  if (cfg->flags & QEVICT_FLAG_ASYNC_ROUTING) {
    e = hipStreamCreateWithFlags(&c->rstream, hipStreamNonBlocking);   // default priority
    const int nl = cfg->num_layers;
    c->route_batch = nl / 2 < 1 ? 1 : (nl / 2 > kRouteBatch ? kRouteBatch : nl / 2);
    c->route_queued.assign(nl, 0);
    c->route_ev_idx.assign(nl, -1);
    c->batch_ev.assign(nl + 1, nullptr);
    c->batch_joined.assign(nl + 1, 0);
    // both streams run on this device: a device-scope release is enough
    const unsigned fl = hipEventDisableTiming | hipEventDisableSystemFence;
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->main_ev, fl);
    for (int i = 0; i <= nl && e == hipSuccess; ++i) e = hipEventCreateWithFlags(&c->batch_ev[i], fl);
    int dev = 0, khz = 0;
    if (e == hipSuccess) e = hipGetDevice(&dev);
    if (e == hipSuccess && (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
                            khz <= 0)) {
      (void)hipGetLastError();
      khz = 100000;                                    // the wall clock's usual 100 MHz
    }
    c->clock_khz = khz;
    c->gate_ticks = (int64_t)(kGateSeconds * 1e3 * khz);
    if (e == hipSuccess)   // sequence 0 and no failure
      e = launch_gate_publish((uint64_t*)(c->ws + kHdrGateSeq), 0, (int32_t*)(c->ws + kHdrGateFail),
                              c->stream);
    if (e != hipSuccess) {
      qevict_cache_destroy(c);
      return hip_fail(e, "creating the routing stream");
    }
  }
  // the fixed scratch of qevict_prefill_scores_noalloc on this (the current)
  // device; if the lookup fails here, that call retries it and reports the error
  if (e == hipSuccess) {
    const char* what = nullptr;
    if (static_obs_scratch(&c->static_scratch, &what) != hipSuccess) {
      c->static_scratch = nullptr;
      (void)hipGetLastError();   // the failed lookup leaves no sticky error behind
    }
  }
  if (e == hipSuccess && cfg->rope_base > 0.f) {
    float* tab = (float*)(c->ws + kHeaderBytes + (int64_t)cfg->num_layers * cfg->batch * c->L.unit_bytes +
                          score_staging_bytes(cfg, c->g));
    const std::vector<float> host = rope_table(cfg);
    e = hipMemcpyAsync(tab, host.data(), host.size() * sizeof(float), hipMemcpyHostToDevice, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);   // the host table goes out of scope
    c->g.rope = tab;
  }
  if (e == hipSuccess && c->rstream) {
    bool beside = false;
    e = routing_fits_beside_attention(c->g, &beside);
    c->queue_wait = (cfg->flags & QEVICT_FLAG_ROUTING_QUEUE_WAIT) ||
                    (!(cfg->flags & QEVICT_FLAG_ROUTING_DEVICE_WAIT) && !beside);
  }
  if (e == hipSuccess) e = launch_init_units(c->g, c->L, c->ws + kHeaderBytes, cfg->num_layers * cfg->batch,
                                   c->stream);
  if (e != hipSuccess) {
    qevict_cache_destroy(c);
    return hip_fail(e, "initialising the cache");
  }
  *out = c;
  return QEVICT_OK;
}

qevict_status qevict_cache_destroy(qevict_cache* c) {
  if (!c) return QEVICT_OK;
  if (c->rstream) {
    (void)flush_routing(c);
    (void)hipStreamSynchronize(c->rstream);
  }
  if (c->main_ev) (void)hipEventDestroy(c->main_ev);
  for (auto e : c->batch_ev)
    if (e) (void)hipEventDestroy(e);
  if (c->rstream) (void)hipStreamDestroy(c->rstream);
  for (auto& t : c->pending) {
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  for (auto e : c->free_events) (void)hipEventDestroy(e);
  delete c;
  return QEVICT_OK;
}

qevict_status qevict_prefill_assign(qevict_cache* c, int32_t layer, const uint16_t* k,
                                    const uint16_t* v, int32_t prompt_len,
                                    const float* init_scores) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  LayerState& ls = c->layers[layer];
  const Geometry& g = c->g;
  if (ls.prefilled) return fail(QEVICT_ERR_BAD_STATE, "layer %d already prefilled", layer);
  const bool key_norm = c->cfg.score_mode == QEVICT_SCORE_KEY_NORM;
  if (prompt_len < g.sink || prompt_len < 1 || prompt_len > c->cfg.max_context)
    return fail(QEVICT_ERR_INVALID_ARG, "prompt_len %d outside [max(1, sink), max_context]", prompt_len);
  const int n_hist = aged_end(g, prompt_len);
  const int n_init = n_started(g, prompt_len);
  // initial scores are read only for the prompt's windows (none when the prompt is all sink)
  if (!k || !v || (!init_scores && !key_norm && n_init > 0))
    return fail(QEVICT_ERR_INVALID_ARG, "null prompt pointer");
  if (((uintptr_t)k & 15) || ((uintptr_t)v & 15))
    return fail(QEVICT_ERR_INVALID_ARG, "prompt keys / values must be 16-byte aligned");
  if (n_hist > kMaxCand)
    return fail(QEVICT_ERR_UNSUPPORTED, "%d prompt windows to route; at most %d", n_hist, kMaxCand);
  if (n_init - n_hist > g.NR)
    return fail(QEVICT_ERR_UNSUPPORTED, "recent region needs more ring slots than configured");

  Geometry gg;
  UnitLayout L;
  uint8_t* base;
  fill_common(c, layer, &gg, &L, &base);
  PackArgs pa{gg, L, base, k, v, prompt_len, 0, g.sink};
  hipError_t e = launch_pack_tokens(pa, c->stream);   // sink tokens
  if (e == hipSuccess) {
    pa.tok0 = g.sink + n_hist * g.W;
    pa.tok1 = prompt_len;
    e = launch_pack_tokens(pa, c->stream);            // tail: recent region and partial window
  }
  float* staging = (float*)(c->ws + kHeaderBytes + (int64_t)c->cfg.num_layers * g.B * c->L.unit_bytes);
  if (key_norm && e == hipSuccess) {
    KeyNormArgs ka{gg, k, prompt_len, n_init, staging};
    e = launch_key_norm_init(ka, c->stream);
    init_scores = staging;
  } else if (c->cfg.score_mode == QEVICT_SCORE_PNORM && e == hipSuccess) {
    ScorePowArgs pa2{init_scores, staging, g.B * n_init, c->cfg.score_p};
    e = launch_score_pow(pa2, c->stream);
    init_scores = staging;
  }
  RetierArgs ra{gg, L, 1, init_scores, n_init, 1, {}};
  ra.unit[0].base = base;
  ra.unit[0].aged_w0 = 0;
  ra.unit[0].aged_w1 = n_hist;
  plan_next(g, c->cfg.max_context, prompt_len + 1, c->cfg.retier_interval, n_hist, &ra.unit[0]);
  if (e == hipSuccess) e = timed(c, 2, c->stream, [&] { return launch_retier(ra, c->stream); });
  MigrateArgs ma{gg, L, 1, {base}, k, v, prompt_len};
  if (e == hipSuccess) e = timed(c, 3, c->stream, [&] { return launch_migrate(ma, g.K_q, g.K_f, c->stream); });
  if (e != hipSuccess) return hip_fail(e, "prefill launch");
  ls.T = prompt_len;
  ls.routed_end = n_hist;
  ls.prefilled = true;
  ls.period_start = true;
  return QEVICT_OK;
}

// ---- initial window scores from the observation queries -------------------
namespace {
constexpr int kObsChunk = 64;   // keys per chunk (one wave) of the observation pass

struct ObsScratch {
  int64_t cml, wl, row_ml, bytes;
};

struct ObsShape {
  int n_w, n_pre, n_chunks;
};

ObsShape obs_shape(const qevict_config* cfg, int32_t prompt_len) {
  ObsShape s;
  const int sink = cfg->sink_tokens, W = cfg->window_tokens;
  s.n_w = prompt_len > sink ? ceil_div(prompt_len - sink, W) : 0;
  s.n_pre = ceil_div(sink, kObsChunk);
  s.n_chunks = s.n_pre + (prompt_len > sink ? ceil_div(prompt_len - sink, kObsChunk) : 0);
  return s;
}

qevict_status obs_check(const qevict_config* cfg, int32_t prompt_len, int32_t n_obs) {
  if (prompt_len < 1 || prompt_len > cfg->max_context)
    return fail(QEVICT_ERR_INVALID_ARG, "prompt_len %d outside [1, max_context]", prompt_len);
  if (n_obs < 1 || n_obs > prompt_len || n_obs > 4096)
    return fail(QEVICT_ERR_INVALID_ARG, "n_obs %d outside [1, min(prompt_len, 4096)]", n_obs);
  return QEVICT_OK;
}

ObsScratch obs_scratch(const qevict_config* cfg, int32_t prompt_len, int32_t n_obs) {
  const int64_t rows = (int64_t)cfg->num_q_heads / cfg->num_kv_heads * n_obs;
  const ObsShape sh = obs_shape(cfg, prompt_len);
  const int64_t bh = (int64_t)cfg->batch * cfg->num_kv_heads;
  ObsScratch s;
  s.cml = 0;
  s.wl = align256(s.cml + 8 * bh * sh.n_chunks * rows);
  s.row_ml = align256(s.wl + 4 * bh * sh.n_w * rows);
  s.bytes = align256(s.row_ml + 8 * bh * rows);
  return s;
}
}  // namespace

qevict_status qevict_prefill_scores_scratch_size(const qevict_config* cfg, int32_t prompt_len,
                                                 int32_t n_obs, size_t* bytes) {
  qevict_status s = check_config(cfg);
  if (s) return s;
  if (!bytes) return fail(QEVICT_ERR_INVALID_ARG, "bytes is NULL");
  if ((s = obs_check(cfg, prompt_len, n_obs))) return s;
  *bytes = (size_t)obs_scratch(cfg, prompt_len, n_obs).bytes;
  return QEVICT_OK;
}

static qevict_status prefill_scores_impl(qevict_cache* c, const uint16_t* q_obs, int32_t n_obs,
                                         const uint16_t* k, int32_t prompt_len, void* scratch,
                                         size_t scratch_bytes, float* scores) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "cache handle is NULL");
  const qevict_config& cfg = c->cfg;
  qevict_status s = obs_check(&cfg, prompt_len, n_obs);
  if (s) return s;
  const Geometry& g = c->g;
  const ObsShape sh = obs_shape(&cfg, prompt_len);
  const int n_w = sh.n_w;
  if (!q_obs || !k || !scratch || (!scores && n_w > 0))
    return fail(QEVICT_ERR_INVALID_ARG, "null pointer");
  if (((uintptr_t)q_obs & 15) || ((uintptr_t)k & 15) || ((uintptr_t)scores & 15))
    return fail(QEVICT_ERR_INVALID_ARG, "queries, keys and scores must be 16-byte aligned");
  if ((uintptr_t)scratch & 255) return fail(QEVICT_ERR_WORKSPACE, "scratch must be 256-byte aligned");
  const ObsScratch L = obs_scratch(&cfg, prompt_len, n_obs);
  if ((int64_t)scratch_bytes < L.bytes)
    return fail(QEVICT_ERR_WORKSPACE, "scratch has %zu bytes, needs %lld", scratch_bytes,
                (long long)L.bytes);
  ObsArgs a;
  a.q = q_obs;
  a.k = k;
  a.B = g.B;
  a.H_q = g.H_q;
  a.H_kv = g.H_kv;
  a.gqa = g.gqa;
  a.T = prompt_len;
  a.n_obs = n_obs;
  a.n_rows = g.gqa * n_obs;
  a.W = g.W;
  a.sink = g.sink;
  a.n_w = n_w;
  a.n_pre = sh.n_pre;
  a.cbase = g.sink - kObsChunk * sh.n_pre;
  a.n_chunks = sh.n_chunks;
  a.n_blk = ceil_div(sh.n_chunks, 4);
  a.scale_log2 = g.scale_log2;
  uint8_t* sb = (uint8_t*)scratch;
  a.cml = (float2*)(sb + L.cml);
  a.wl = (float*)(sb + L.wl);
  a.row_ml = (float2*)(sb + L.row_ml);
  a.scores = scores;
  const hipError_t e = timed(c, 4, c->stream, [&] { return launch_prefill_scores(a, c->stream); });
  if (e != hipSuccess) return hip_fail(e, "prefill_scores launch");
  return QEVICT_OK;
}

qevict_status qevict_prefill_scores(qevict_cache* c, const uint16_t* q_obs, int32_t n_obs,
                                    const uint16_t* k, int32_t prompt_len, void* scratch,
                                    size_t scratch_bytes, float* scores) {
  return prefill_scores_impl(c, q_obs, n_obs, k, prompt_len, scratch, scratch_bytes, scores);
}

qevict_status qevict_prefill_scores_noalloc(qevict_cache* c, const uint16_t* q_obs, int32_t n_obs,
                                            const uint16_t* k, int32_t prompt_len, float* scores) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "cache handle is NULL");
  qevict_status s = obs_check(&c->cfg, prompt_len, n_obs);
  if (s) return s;
  const int64_t need = obs_scratch(&c->cfg, prompt_len, n_obs).bytes;
  if (need > kStaticObsScratchBytes)
    return fail(QEVICT_ERR_WORKSPACE,
                "this prompt needs %lld bytes of scratch; the fixed scratch holds %lld "
                "(use qevict_prefill_scores with a caller buffer)",
                (long long)need, (long long)kStaticObsScratchBytes);
  if (!c->static_scratch) {
    const char* what = "lookup";
    const hipError_t e = static_obs_scratch(&c->static_scratch, &what);
    if (e != hipSuccess) {
      c->static_scratch = nullptr;
      return fail(QEVICT_ERR_DEVICE, "fixed scratch address (%s): %s", what, hipGetErrorString(e));
    }
  }
  return prefill_scores_impl(c, q_obs, n_obs, k, prompt_len, c->static_scratch,
                             (size_t)kStaticObsScratchBytes, scores);
}

qevict_status qevict_decode_attend(qevict_cache* c, int32_t layer, const uint16_t* q,
                                   const uint16_t* k_new, const uint16_t* v_new, void* out) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  LayerState& ls = c->layers[layer];
  const Geometry& g = c->g;
  if (!ls.prefilled) return fail(QEVICT_ERR_BAD_STATE, "layer %d not prefilled", layer);
  if (!q || !k_new || !v_new || !out) return fail(QEVICT_ERR_INVALID_ARG, "null pointer");
  if (((uintptr_t)q & 15) || ((uintptr_t)k_new & 15))
    return fail(QEVICT_ERR_INVALID_ARG, "q and k_new must be 16-byte aligned");
  if (ls.T + 1 > c->cfg.max_context)
    return fail(QEVICT_ERR_BAD_STATE, "max_context %d reached", c->cfg.max_context);
  const int T = ls.T + 1;
  const int n_ring = n_started(g, T) - ls.routed_end;
  if (n_ring > g.NR)
    return fail(QEVICT_ERR_BAD_STATE, "%d unrouted windows exceed the ring (%d); call retier", n_ring,
                g.NR);
  AttnArgs a;
  fill_common(c, layer, &a.g, &a.L, &a.base);
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.out = out;
  a.T = T;
  a.ring_w0 = ls.routed_end;
  a.n_ring = n_ring;
  a.n_sink_items = g.NS;
  a.decay = (c->cfg.score_mode == QEVICT_SCORE_DECAY && ls.period_start) ? c->cfg.score_decay : 1.0f;
  a.key_norm = c->cfg.score_mode == QEVICT_SCORE_KEY_NORM;
  a.pnorm_p = c->cfg.score_mode == QEVICT_SCORE_PNORM ? c->cfg.score_p : 0.f;
  a.period_start = ls.period_start;
  hipError_t e = hipSuccess;
  if (g.flags & QEVICT_FLAG_DEBUG_MASSES) {
    for (int b = 0; b < g.B && e == hipSuccess; ++b)
      e = hipMemsetAsync(unit_base(c, layer, b) + c->L.dbg_mass, 0, 4LL * g.H_q * (g.nwc + 1),
                         c->stream);
  }
  if (e == hipSuccess) e = timed(c, 0, c->stream, [&] { return launch_attend(a, c->stream); });
  if (e == hipSuccess) e = timed(c, 1, c->stream, [&] { return launch_merge(a, c->stream); });
  if (e != hipSuccess) return hip_fail(e, "decode_attend launch");
  ls.T = T;
  ls.period_start = false;
  return QEVICT_OK;
}

qevict_status qevict_retier(qevict_cache* c, int32_t layer, qevict_retier_stats* stats) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  LayerState& ls = c->layers[layer];
  const Geometry& g = c->g;
  if (!ls.prefilled) return fail(QEVICT_ERR_BAD_STATE, "layer %d not prefilled", layer);
  const int a1 = aged_end(g, ls.T);
  const int a0 = ls.routed_end;
  Geometry gg;
  UnitLayout L;
  uint8_t* base;
  fill_common(c, layer, &gg, &L, &base);
  RetierUnit unit{};
  unit.base = base;
  unit.aged_w0 = a0;
  unit.aged_w1 = a1 > a0 ? a1 : a0;
  plan_next(g, c->cfg.max_context, ls.T + 1, c->cfg.retier_interval, unit.aged_w1, &unit);
  // grid of the migration launch: sized for the windows a routing event usually
  // moves (a few per step between events); larger events loop inside the kernel
  const int max_q = std::min(std::max(g.K_q, g.K_f), 4 * c->cfg.retier_interval);
  hipError_t e = hipSuccess;
  if (c->rstream) {
    // asynchronous routing: queue the request; a batch is launched on the
    // routing stream once it is full (or the layer is needed again); a layer
    // queued already goes to the next batch
    if (c->route_queued[layer] && (e = flush_routing(c)) != hipSuccess) return hip_fail(e, "retier launch");
    c->route_queue.push_back(RouteRequest{layer, unit, max_q, max_q});
    c->route_queued[layer] = 1;
    if (stats || (int)c->route_queue.size() >= c->route_batch) e = flush_routing(c);
  } else {
    RetierArgs ra{gg, L, 0, nullptr, 0, 1, {unit}};
    MigrateArgs ma{gg, L, 1, {base}, nullptr, nullptr, 0};
    e = timed(c, 2, c->stream, [&] { return launch_retier(ra, c->stream); });
    if (e == hipSuccess) e = timed(c, 3, c->stream, [&] { return launch_migrate(ma, max_q, max_q, c->stream); });
  }
  if (e != hipSuccess) return hip_fail(e, "retier launch");
  if (a1 > a0) ls.routed_end = a1;
  ls.period_start = true;
  if (stats) {
    memset(stats, 0, sizeof *stats);
    if ((e = join_layer(c, layer)) != hipSuccess) return hip_fail(e, "joining the routing stream");
    for (int b = 0; b < g.B; ++b) {
      int32_t st[ST_N];
      e = hipMemcpyAsync(st, unit_base(c, layer, b) + c->L.stats, sizeof st, hipMemcpyDeviceToHost,
                         c->stream);
      if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
      if (e != hipSuccess) return hip_fail(e, "reading retier stats");
      stats->promotions += st[ST_PROMO];
      stats->admissions_full += st[ST_ADMIT];
      stats->first_quantizations += st[ST_FIRSTQ];
      stats->reactivations += st[ST_REACT];
      stats->evictions += st[ST_EVICT];
      stats->n_full += st[ST_NF];
      stats->n_quant_int4 += st[ST_NQ4];
      stats->n_quant_int2 += st[ST_NQ2];
    }
    return device_errors(c, layer);
  }
  return QEVICT_OK;
}

static qevict_status read_window_state(qevict_cache* c, int layer, int seq, int window, int8_t* tier,
                                       int8_t* led) {
  uint8_t* ub = unit_base(c, layer, seq);
  hipError_t e = hipMemcpyAsync(tier, ub + c->L.tier + window, 1, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(led, ub + c->L.ledger + window, 1, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  return e == hipSuccess ? QEVICT_OK : hip_fail(e, "reading window state");
}

static qevict_status manual_move(qevict_cache* c, int layer, int seq, int window, int to_quant) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  const Geometry& g = c->g;
  if (!c->layers[layer].prefilled) return fail(QEVICT_ERR_BAD_STATE, "layer not prefilled");
  if (seq < 0 || seq >= g.B) return fail(QEVICT_ERR_INVALID_ARG, "seq %d out of range", seq);
  if (window < 0 || window >= g.nwc) return fail(QEVICT_ERR_INVALID_ARG, "window %d out of range", window);
  if ((s = device_errors(c, layer))) return s;
  int8_t tier = 0, led = 0;
  if ((s = read_window_state(c, layer, seq, window, &tier, &led))) return s;
  if (tier != (to_quant ? T_FULL : T_QUANT))
    return fail(QEVICT_ERR_BAD_STATE, "window %d is not in the %s tier", window,
                to_quant ? "Full" : "Quantized");
  if (!to_quant && (g.flags & QEVICT_FLAG_NO_PROMOTION))
    return fail(QEVICT_ERR_BAD_STATE, "promotion disabled by QEVICT_FLAG_NO_PROMOTION");
  // tier occupancy
  std::vector<int8_t> tiers(g.nwc);
  hipError_t e = hipMemcpyAsync(tiers.data(), unit_base(c, layer, seq) + c->L.tier, g.nwc,
                                hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "reading tiers");
  int nf = 0, nq = 0;
  for (int8_t t : tiers) {
    nf += t == T_FULL;
    nq += t == T_QUANT;
  }
  if (to_quant && nq >= g.K_q) return fail(QEVICT_ERR_CAPACITY, "Quantized tier holds K_q windows");
  if (!to_quant && nf >= g.K_f) return fail(QEVICT_ERR_CAPACITY, "Full tier holds K_f windows");
  Geometry gg;
  UnitLayout L;
  uint8_t* base;
  fill_common(c, layer, &gg, &L, &base);
  RetierArgs ra{gg, L, 0, nullptr, 0, 1, {}};
  ra.unit[0].base = base;
  // the migration kernels read work lists per sequence: run them on this sequence only
  Geometry one = gg;
  one.B = 1;
  MigrateArgs ma{one, L, 1, {unit_base(c, layer, seq)}, nullptr, nullptr, 0};
  e = launch_manual_move(ra, seq, window, to_quant, c->stream);
  if (e == hipSuccess) e = launch_migrate(ma, 1, 1, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "manual move");
  return device_errors(c, layer);
}

qevict_status qevict_quantize_window(qevict_cache* c, int32_t layer, int32_t seq, int32_t window) {
  return manual_move(c, layer, seq, window, 1);
}

qevict_status qevict_promote_window(qevict_cache* c, int32_t layer, int32_t seq, int32_t window) {
  return manual_move(c, layer, seq, window, 0);
}

qevict_status qevict_get_state(qevict_cache* c, int32_t layer, int32_t seq, int8_t* tiers,
                               float* scores, int8_t* ledger, int8_t* bits, int32_t cap,
                               int32_t* n_windows) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  const Geometry& g = c->g;
  if (seq < 0 || seq >= g.B) return fail(QEVICT_ERR_INVALID_ARG, "seq %d out of range", seq);
  if (cap < 0) return fail(QEVICT_ERR_INVALID_ARG, "cap < 0");
  const LayerState& ls = c->layers[layer];
  const int nst = n_started(g, ls.T);
  const int n = nst < cap ? nst : cap;
  if (n_windows) *n_windows = nst;
  uint8_t* ub = unit_base(c, layer, seq);
  hipError_t e = hipSuccess;
  if (tiers && n) e = hipMemcpyAsync(tiers, ub + c->L.tier, n, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess && scores && n)
    e = hipMemcpyAsync(scores, ub + c->L.score, 4LL * n, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess && ledger && n)
    e = hipMemcpyAsync(ledger, ub + c->L.ledger, n, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess && bits && n)
    e = hipMemcpyAsync(bits, ub + c->L.bits, n, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "get_state copy");
  if (tiers)
    for (int w = ls.routed_end; w < n; ++w) tiers[w] = T_OPEN;   // recent region / not yet routed
  return device_errors(c, layer);
}

qevict_status qevict_memory_report(qevict_cache* c, int32_t layer, int32_t seq, qevict_memory* out) {
  if (!out) return fail(QEVICT_ERR_INVALID_ARG, "out is NULL");
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  const Geometry& g = c->g;
  std::vector<int8_t> tiers(g.nwc), ledger(g.nwc), bits(g.nwc);
  int32_t n = 0;
  s = qevict_get_state(c, layer, seq, tiers.data(), nullptr, ledger.data(), bits.data(), g.nwc, &n);
  if (s) return s;
  const int64_t T = c->layers[layer].T, Hkv = g.H_kv, d = g.d, W = g.W, G = g.G;
  const int64_t tok = 4 * Hkv * d;   // bf16 key and value of one token
  const int64_t meta = 4 * Hkv * d + 4 * Hkv * W * (d / G);
  int64_t routed = 0;
  qevict_memory m{};
  m.sink = tok * std::min<int64_t>(g.sink, T);
  for (int w = 0; w < n; ++w) {
    const int t = tiers[w];
    if (t == T_FULL || t == T_QUANT || t == T_EVICTED) ++routed;
    const int64_t codes = 2 * Hkv * W * d * bits[w] / 8;
    if (t == T_FULL) {
      m.full += tok * W;
      m.position += 8;
    } else if (t == T_QUANT) {
      m.quant_codes += codes;
      m.quant_meta += meta;
      m.position += 8;
    }
    if (ledger[w] == L_DORMANT) m.ledger += codes + meta;
    if (ledger[w] != L_NONE) m.ledger += 2;
  }
  m.recent = tok * std::max<int64_t>(0, T - g.sink - W * routed);
  m.total = m.sink + m.recent + m.full + m.quant_codes + m.quant_meta + m.position + m.ledger;
  *out = m;
  return QEVICT_OK;
}

qevict_status qevict_export_window(qevict_cache* c, int32_t layer, int32_t seq, int32_t window,
                                   uint8_t* codes_k, uint8_t* codes_v, uint16_t* meta_k,
                                   uint16_t* meta_v, uint16_t* full_k, uint16_t* full_v) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  const Geometry& g = c->g;
  if (seq < 0 || seq >= g.B) return fail(QEVICT_ERR_INVALID_ARG, "seq %d out of range", seq);
  if (window < 0 || window >= g.nwc) return fail(QEVICT_ERR_INVALID_ARG, "window out of range");
  uint8_t* ub = unit_base(c, layer, seq);
  int8_t tier, led, nb;
  int32_t fs, qs;
  hipError_t e = hipMemcpyAsync(&tier, ub + c->L.tier + window, 1, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipMemcpyAsync(&led, ub + c->L.ledger + window, 1, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipMemcpyAsync(&nb, ub + c->L.bits + window, 1, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipMemcpyAsync(&fs, ub + c->L.fslot + 4LL * window, 4, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipMemcpyAsync(&qs, ub + c->L.qslot + 4LL * window, 4, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "export_window state");
  const int W = g.W, d = kHeadDim, ng = d / g.G;
  const bool want_q = codes_k || codes_v || meta_k || meta_v;
  const bool want_f = full_k || full_v;
  if (want_q && (led == L_NONE || qs < 0)) return fail(QEVICT_ERR_BAD_STATE, "window has no ledger");
  if (want_f && (tier != T_FULL || fs < 0)) return fail(QEVICT_ERR_BAD_STATE, "window is not Full");
  std::vector<uint8_t> rec(g.qslot_bytes), slot(g.fslot_bytes);
  if (want_q)
    e = hipMemcpyAsync(rec.data(), ub + c->L.qpool + (int64_t)qs * g.qslot_bytes, g.qslot_bytes,
                       hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess && want_f)
    e = hipMemcpyAsync(slot.data(), ub + c->L.fpool + (int64_t)fs * g.fslot_bytes, g.fslot_bytes,
                       hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "export_window copy");
  for (int h = 0; h < g.H_kv; ++h) {
    const uint8_t* r = rec.data() + h * g.qrec_bytes;
    const uint8_t* f = slot.data() + h * g.fhead_bytes;
    for (int t = 0; t < W; ++t)
      for (int ch = 0; ch < d; ++ch) {
        const int64_t o = ((int64_t)h * W + t) * d + ch;
        int ee, L, j, sh;
        int64_t off;
        if (codes_k) {
          if (W == 8) {
            code_loc8(nb, 0, t, ch, &off, &sh);
          } else {
            k_code_pos(t, ch, &ee, &L, &j);
            code_loc(nb, ee, L, j, &off, &sh);
          }
          uint32_t w32;
          memcpy(&w32, r + off, 4);
          codes_k[o] = (uint8_t)((w32 >> sh) & ((1u << nb) - 1));
        }
        if (codes_v) {
          if (W == 8) {
            code_loc8(nb, 1, t, ch, &off, &sh);
          } else {
            v_code_pos(t, ch, &ee, &L, &j);
            code_loc(nb, ee, L, j, &off, &sh);
          }
          uint32_t w32;
          memcpy(&w32, r + g.qcodes_bytes + off, 4);
          codes_v[o] = (uint8_t)((w32 >> sh) & ((1u << nb) - 1));
        }
        if (full_k) memcpy(full_k + o, f + k_elem_off(W, t, ch), 2);
        if (full_v) memcpy(full_v + o, f + v_elem_off(W, t, ch), 2);
      }
    if (meta_k) {   // [h][2][d]: one key group per channel
      memcpy(meta_k + (int64_t)h * 2 * d, r + meta_k_off(g), 2 * d);
      memcpy(meta_k + (int64_t)h * 2 * d + d, r + meta_k_off(g) + 2 * d, 2 * d);
    }
    if (meta_v) {   // [h][2][W][d/G]
      for (int t = 0; t < W; ++t)
        for (int vg = 0; vg < ng; ++vg) {
          const int64_t mo = meta_v_elem(g, t, vg);
          memcpy(meta_v + ((int64_t)h * 2 * W + t) * ng + vg, r + mo, 2);
          memcpy(meta_v + ((int64_t)h * 2 * W + W + t) * ng + vg, r + mo + meta_v_zero_delta(g), 2);
        }
    }
  }
  return QEVICT_OK;
}

qevict_status qevict_debug_shift_keys(qevict_cache* c, int32_t layer, int32_t seq, int32_t window,
                                      const float* delta) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  const Geometry& g = c->g;
  if (seq < 0 || seq >= g.B || window < 0 || window >= g.nwc || !delta)
    return fail(QEVICT_ERR_INVALID_ARG, "seq / window / delta");
  uint8_t* ub = unit_base(c, layer, seq);
  int8_t led;
  int32_t qs;
  hipError_t e = hipMemcpyAsync(&led, ub + c->L.ledger + window, 1, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipMemcpyAsync(&qs, ub + c->L.qslot + 4LL * window, 4, hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e, "shift_keys state");
  if (led == L_NONE || qs < 0) return fail(QEVICT_ERR_BAD_STATE, "window has no ledger");
  const int d = kHeadDim;
  std::vector<uint16_t> z(d);
  for (int h = 0; h < g.H_kv; ++h) {
    uint8_t* zp = ub + c->L.qpool + (int64_t)qs * g.qslot_bytes + h * g.qrec_bytes + meta_k_off(g) + 2 * d;
    e = hipMemcpyAsync(z.data(), zp, 2 * d, hipMemcpyDeviceToHost, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return hip_fail(e, "shift_keys read");
    for (int ch = 0; ch < d; ++ch)
      z[ch] = host_rne_fp16(host_fp16_to_double(z[ch]) + (double)delta[h * d + ch]);
    e = hipMemcpyAsync(zp, z.data(), 2 * d, hipMemcpyHostToDevice, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return hip_fail(e, "shift_keys write");
  }
  return QEVICT_OK;
}

qevict_status qevict_debug_masses(qevict_cache* c, int32_t layer, float* masses, int32_t n_cap) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  const Geometry& g = c->g;
  if (!(g.flags & QEVICT_FLAG_DEBUG_MASSES))
    return fail(QEVICT_ERR_BAD_STATE, "cache created without QEVICT_FLAG_DEBUG_MASSES");
  if (!masses || n_cap != g.nwc) return fail(QEVICT_ERR_INVALID_ARG, "n_cap must equal %d", g.nwc);
  for (int b = 0; b < g.B; ++b) {
    hipError_t e = hipMemcpyAsync(masses + (int64_t)b * g.H_q * (g.nwc + 1),
                                  unit_base(c, layer, b) + c->L.dbg_mass, 4LL * g.H_q * (g.nwc + 1),
                                  hipMemcpyDeviceToHost, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return hip_fail(e, "debug masses");
  }
  return QEVICT_OK;
}

qevict_status qevict_debug_last_masses(qevict_cache* c, int32_t layer, float* masses) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  return qevict_debug_masses(c, layer, masses, c->g.nwc);
}

qevict_status qevict_routing_order(qevict_cache* c, int32_t* order) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "cache is NULL");
  if (!order) return fail(QEVICT_ERR_INVALID_ARG, "order is NULL");
  *order = !c->rstream ? QEVICT_ROUTING_SYNC : c->queue_wait ? QEVICT_ROUTING_QUEUE_WAIT : QEVICT_ROUTING_GATE;
  return QEVICT_OK;
}

qevict_status qevict_debug_routing_gate(qevict_cache* c, int64_t timeout_us, int32_t release) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "cache is NULL");
  if (!c->rstream || c->queue_wait)
    return fail(QEVICT_ERR_INVALID_ARG, "the cache orders no routing with the device-side wait");
  if (timeout_us <= 0) return fail(QEVICT_ERR_INVALID_ARG, "timeout_us must be positive");
  if (hipError_t e = flush_routing(c)) return hip_fail(e, "launching queued routing");
  c->gate_ticks = timeout_us * c->clock_khz / 1000;
  c->gate_release = release != 0;
  return QEVICT_OK;
}

qevict_status qevict_profile_enable(qevict_cache* c, int32_t on) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "cache is NULL");
  fold_pending(c);
  c->profiling = on != 0;
  for (int i = 0; i < kNumTimed; ++i) {
    c->prof_ms[i] = 0;
    c->prof_n[i] = 0;
  }
  return QEVICT_OK;
}

qevict_status qevict_profile_read(qevict_cache* c, int32_t kernel, double* total_ms, int64_t* count) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "cache is NULL");
  if (kernel < 0 || kernel >= kNumTimed) return fail(QEVICT_ERR_INVALID_ARG, "kernel id");
  fold_pending(c);
  if (total_ms) *total_ms = c->prof_ms[kernel];
  if (count) *count = c->prof_n[kernel];
  return QEVICT_OK;
}

qevict_status qevict_join_routing(qevict_cache* c) {
  if (!c) return fail(QEVICT_ERR_INVALID_ARG, "cache is NULL");
  if (!c->rstream) return QEVICT_OK;
  if (hipError_t e = flush_routing(c)) return hip_fail(e, "launching queued routing");
  for (int l = 0; l < c->cfg.num_layers; ++l)
    if (hipError_t e = join_layer(c, l)) return hip_fail(e, "joining the routing stream");
  return QEVICT_OK;
}

qevict_status qevict_last_attend_bytes(qevict_cache* c, int32_t layer, int64_t* bytes) {
  qevict_status s = check_handle(c, layer);
  if (s) return s;
  if (!bytes) return fail(QEVICT_ERR_INVALID_ARG, "bytes is NULL");
  const Geometry& g = c->g;
  const LayerState& ls = c->layers[layer];
  int64_t total = 0;
  for (int b = 0; b < g.B; ++b) {
    int32_t st[ST_N];
    hipError_t e = hipMemcpyAsync(st, unit_base(c, layer, b) + c->L.stats, sizeof st,
                                  hipMemcpyDeviceToHost, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return hip_fail(e, "reading tier sizes");
    const int64_t per_f = g.fslot_bytes;
    const int64_t meta = (int64_t)g.H_kv * (4 * kHeadDim + (int64_t)g.W * (kHeadDim / g.G) * 4);
    const int64_t per_q4 = (int64_t)g.H_kv * 2 * g.W * kHeadDim * 4 / 8 + meta;
    const int64_t per_q2 = (int64_t)g.H_kv * 2 * g.W * kHeadDim * 2 / 8 + meta;
    const int recent_tok = ls.T - g.sink - ls.routed_end * g.W;
    const int64_t tok_bytes = (int64_t)2 * g.H_kv * kHeadDim * 2;
    total += st[ST_NF] * per_f + st[ST_NQ4] * per_q4 + st[ST_NQ2] * per_q2 +
             (int64_t)(recent_tok + g.sink) * tok_bytes +
             (int64_t)2 * g.H_q * kHeadDim * 2 +                  // q in, out (bf16 equivalent)
             (int64_t)(st[ST_NF] + st[ST_NQ4] + st[ST_NQ2] + n_started(g, ls.T) - ls.routed_end) * 8;
  }
  *bytes = total;
  return QEVICT_OK;
}

}  // extern "C"
