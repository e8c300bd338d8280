// moe_ffn_forward: routing, dispatch, per-stage GEMM selection and the
// expert pipeline over HIP streams.
//
// Streams (per device, created once, default priority):
//   caller stream s0 : route, dispatch indices, the host copy of counts
//   sg (gather)      : stage i's row gather (the one-GPU stand-in for the
//                      dispatch all2all of one stage)
//   sm (GEMM)        : shared experts, then each stage's expert GEMMs
//   sc (combine)     : each stage's weighted combine, in stage order
// With one stage and shared experts only the shared FFN leaves the caller's
// stream: the routed GEMMs and the combine follow the dispatch on s0.
// Stage i's GEMMs wait for its gather; its combine waits for its GEMMs, so
// gather(i+1) and combine(i-1) overlap GEMM(i).  By default a stage is an
// expert group: local experts [i*EL/PN, (i+1)*EL/PN), whose rows are one
// contiguous range of the expert-sorted buffers, so each expert's weights
// are read by exactly one stage (the paper's horizontal split with weights
// split by expert, Sec. 4.3).  With token-range stages the dispatch orders
// rows by (stage, expert, token) instead, so stage i's rows are again one
// contiguous range, now covering every expert.  The GEMM kind of each stage
// is chosen from its row counts (GroupGemm for small loads, DenseGemm per
// expert for large ones).
#include <algorithm>
#include <cmath>
#include <map>
#include <memory>
#include <mutex>
#include <vector>

#include <cstdio>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "common.h"

namespace moe {
namespace {

// The routed GEMMs run beside the shared FFN (one stage) up to this many
// tokens.
constexpr int64_t kRoutedBesideSharedMaxTokens = 4096;

// AUTO weighs GroupGemm against DenseGemm with the launch-cost model only
// for stages of at most this many experts: every dense launch pays its own
// partial round of tiles, so with more experts per stage the single grouped
// launch wins at every load the model (and the measured sweep) covers, and
// AUTO then needs no host copy of the row counts.
constexpr int kAutoDenseMaxExperts = 2;

enum Phase {
    PH_ROUTE, PH_PERMUTE, PH_GATHER, PH_GATEUP, PH_DOWN, PH_SHARED, PH_COMBINE, PH_TOTAL, PH_N
};

// Per-device state of moe_ffn_forward: three side streams and the pinned
// host copy of the row counts.  `call` is held for a whole call, so two
// host threads driving the same device take turns (their enqueues do not
// interleave on the shared streams, events and pinned buffer).
struct Streams {
    hipStream_t sg = nullptr, sm = nullptr, sc = nullptr;
};
struct DevState {
    std::mutex call;
    Streams plain;                     // no CU masks
    std::map<int, Streams> masked;     // by side_cus: sg, sc on those CUs, sm on the rest
    std::vector<hipEvent_t> sync_ev;   // ordering events (no timing)
    int32_t *pinned_counts = nullptr;  // host-visible copy of counts
    bool ready = false;
};

std::mutex g_mu;  // guards g_dev and the creation of each device's state
std::vector<std::unique_ptr<DevState>> g_dev;

moe_status ensure_events(std::vector<hipEvent_t> &pool, size_t n, unsigned flags) {
    while (pool.size() < n) {
        hipEvent_t e;
        MOE_HIP(hipEventCreateWithFlags(&e, flags));
        pool.push_back(e);
    }
    return MOE_OK;
}

moe_status get_state(DevState **out) {
    int dev = 0;
    MOE_HIP(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lock(g_mu);
    if ((int)g_dev.size() <= dev) g_dev.resize(dev + 1);
    if (!g_dev[dev]) g_dev[dev].reset(new DevState);
    DevState &st = *g_dev[dev];
    if (!st.ready) {
        MOE_HIP(hipStreamCreateWithFlags(&st.plain.sg, hipStreamNonBlocking));
        MOE_HIP(hipStreamCreateWithFlags(&st.plain.sm, hipStreamNonBlocking));
        MOE_HIP(hipStreamCreateWithFlags(&st.plain.sc, hipStreamNonBlocking));
        MOE_HIP(hipHostMalloc((void **)&st.pinned_counts, sizeof(int32_t) * kMaxExperts,
                              hipHostMallocDefault));
        st.ready = true;
    }
    *out = &st;
    return MOE_OK;
}

// CU masks: the first `side` CUs of the mask for the gather and combine
// streams, the others for the GEMM stream.  The driver deals a queue's mask
// bits round-robin over the XCDs and, inside an XCD, over its shader
// engines, so the first n bits take the same number of CUs from every XCD
// and engine.  (Measured: a mask that took the side CUs from one engine per
// XCD left that engine half of its CUs for an equal share of the GEMM's
// workgroups and doubled the GEMM time.)
void side_cu_masks(int side, int cus, std::vector<uint32_t> &side_mask,
                   std::vector<uint32_t> &gemm_mask) {
    const int words = (cus + 31) / 32;
    side_mask.assign(words, 0u);
    gemm_mask.assign(words, 0u);
    for (int c = 0; c < cus; ++c) {
        if (c < side) side_mask[c / 32] |= 1u << (c % 32);
        else gemm_mask[c / 32] |= 1u << (c % 32);
    }
}

// Streams of a call: the plain ones, or (side > 0) the set whose gather and
// combine streams run on `side` CUs and whose GEMM stream runs on the rest
// (created once per device and side count, default priority).
moe_status get_streams(DevState *st, int side, Streams *out) {
    if (side <= 0) {
        *out = st->plain;
        return MOE_OK;
    }
    std::lock_guard<std::mutex> lock(g_mu);
    auto it = st->masked.find(side);
    if (it == st->masked.end()) {
        std::vector<uint32_t> sm_mask, gm_mask;
        side_cu_masks(side, device_cu_count(), sm_mask, gm_mask);
        Streams s;
        MOE_HIP(hipExtStreamCreateWithCUMask(&s.sg, (uint32_t)sm_mask.size(), sm_mask.data()));
        MOE_HIP(hipExtStreamCreateWithCUMask(&s.sc, (uint32_t)sm_mask.size(), sm_mask.data()));
        MOE_HIP(hipExtStreamCreateWithCUMask(&s.sm, (uint32_t)gm_mask.size(), gm_mask.data()));
        it = st->masked.emplace(side, s).first;
    }
    *out = it->second;
    return MOE_OK;
}

struct TimedSpan {
    int phase;
    hipEvent_t start, stop;
};

struct TimingRecord {
    std::vector<TimedSpan> spans;
    int gateup_launches = 0, down_launches = 0, dense_stages = 0, group_stages = 0;
    int pipeline_n = 0;
    int calls = 0;       // timed calls in the record
    int device = -1;     // device of the record's events
    size_t events = 0;   // events of the pool in use by the record
    bool valid = false;
    bool read = false;   // returned by moe_last_timing: the next timed call starts anew
};
thread_local TimingRecord g_timing;
// timing events of the calling thread, per device: a thread's last timed
// call stays readable whatever other threads do
thread_local std::vector<std::vector<hipEvent_t>> t_time_ev;

// Records spans into the calling thread's record when enabled: every
// phase (MOE_FLAG_TIMING), or only the GEMM phases (MOE_FLAG_TIMING_GEMM).
// A span that starts on the stream where the previous span just ended, with
// nothing enqueued in between, reuses that span's stop event as its start.
class Timer {
   public:
    Timer(std::vector<hipEvent_t> *pool, int flags)
        : pool_(pool), all_((flags & MOE_FLAG_TIMING) != 0),
          gemm_((flags & (MOE_FLAG_TIMING | MOE_FLAG_TIMING_GEMM)) != 0),
          used_(g_timing.events) {}
    ~Timer() { g_timing.events = used_; }
    // Starts a span of `phase` on stream s; returns its index (or -1).
    moe_status begin(hipStream_t s, int phase, int *idx = nullptr) {
        int &i = idx ? *idx : cur_;
        i = -1;
        if (!timed(phase)) {
            chain_ = false;
            return MOE_OK;
        }
        hipEvent_t a, b;
        // (the caller's stream may be the null stream: compare only after a
        // span has ended)
        const bool chain = chain_ && last_s_ == s;
        MOE_TRY(ensure_events(*pool_, used_ + 2, hipEventDefault));
        a = chain ? last_stop_ : (*pool_)[used_];
        b = (*pool_)[used_ + 1];
        used_ += 2;
        if (!chain) MOE_HIP(hipEventRecord(a, s));
        chain_ = false;
        i = (int)g_timing.spans.size();
        g_timing.spans.push_back({phase, a, b});
        return MOE_OK;
    }
    moe_status end(hipStream_t s, int idx = -2) {
        const int i = idx == -2 ? cur_ : idx;
        if (i < 0) return MOE_OK;
        MOE_HIP(hipEventRecord(g_timing.spans[i].stop, s));
        chain_ = true;
        last_s_ = s;
        last_stop_ = g_timing.spans[i].stop;
        return MOE_OK;
    }
    // Something else was enqueued: the next span records its own start.
    void gap() { chain_ = false; }

   private:
    bool timed(int phase) const {
        return all_ || (gemm_ && (phase == PH_GATEUP || phase == PH_DOWN || phase == PH_SHARED));
    }
    std::vector<hipEvent_t> *pool_;
    bool all_, gemm_;
    size_t used_;
    int cur_ = -1;
    bool chain_ = false;  // the last enqueue was a span's stop event
    hipStream_t last_s_ = nullptr;
    hipEvent_t last_stop_ = nullptr;
};

moe_status check_opts(const moe_dims *d, const moe_opts *o) {
    if (o->gemm_mode < MOE_GEMM_AUTO || o->gemm_mode > MOE_GEMM_DENSE)
        return fail(MOE_ERR_INVALID, "gemm_mode %d unknown", o->gemm_mode);
    if (o->dense_min_rows < 0) return fail(MOE_ERR_INVALID, "dense_min_rows < 0");
    if (o->chunk_mode != MOE_CHUNK_EXPERTS && o->chunk_mode != MOE_CHUNK_TOKENS)
        return fail(MOE_ERR_INVALID, "chunk_mode %d unknown", o->chunk_mode);
    if (o->pipeline_n < 0) return fail(MOE_ERR_INVALID, "pipeline_n %d < 0", o->pipeline_n);
    if (o->pipeline_n == 0 && o->chunk_mode != MOE_CHUNK_EXPERTS)
        return fail(MOE_ERR_INVALID, "pipeline_n 0 (chosen by the library) needs expert stages");
    if (o->chunk_mode == MOE_CHUNK_EXPERTS && o->pipeline_n > 0 &&
        d->local_count % o->pipeline_n)
        return fail(MOE_ERR_INVALID, "pipeline_n %d must divide local_count %d",
                    o->pipeline_n, d->local_count);
    if (o->chunk_mode == MOE_CHUNK_TOKENS &&
        (int64_t)o->pipeline_n * d->local_count > kMaxExperts)
        return fail(MOE_ERR_UNSUPPORTED, "token stages: pipeline_n * local_count > %d",
                    kMaxExperts);
    if (o->gemm_cu_budget < 0) return fail(MOE_ERR_INVALID, "gemm_cu_budget < 0");
    if (o->flags &
        ~(MOE_FLAG_TIMING | MOE_FLAG_TIMING_GEMM | MOE_FLAG_EXACT_ORDER | MOE_FLAG_SERIAL))
        return fail(MOE_ERR_INVALID, "unknown flags 0x%x", o->flags);
    if (o->dense_tile_rows != 0 && !valid_tile_rows(o->dense_tile_rows))
        return fail(MOE_ERR_INVALID, "dense_tile_rows %d is not 0, 128, 192, 256 or 320",
                    o->dense_tile_rows);
    if (o->side_cus < 0 || o->side_cus > kMaxExperts - 8)
        return fail(MOE_ERR_INVALID, "side_cus %d outside [0, 248]", o->side_cus);
    if (o->group_tile_rows != 0 && !valid_tile_rows(o->group_tile_rows))
        return fail(MOE_ERR_INVALID, "group_tile_rows %d is not 0, 128, 192, 256 or 320",
                    o->group_tile_rows);
    return MOE_OK;
}

}  // namespace

int forward_buckets(const moe_dims *d, const moe_opts *o) {
    if (check_opts(d, o) != MOE_OK) return 0;
    return o->chunk_mode == MOE_CHUNK_TOKENS ? o->pipeline_n * d->local_count : d->local_count;
}

// Experts per pipeline stage.
int stage_experts(const moe_dims &d, const moe_opts &o) {
    if (o.chunk_mode == MOE_CHUNK_TOKENS) return d.local_count;
    return o.pipeline_n > 0 ? d.local_count / o.pipeline_n : 1;
}

bool needs_host_counts(const moe_dims &d, const moe_opts &o) {
    // row counts are needed on the host to size per-expert dense launches and
    // stage gathers, and for AUTO to weigh the two GEMM kinds: with a fixed
    // threshold only when some expert can reach it (an expert has at most T
    // rows), with the cost model only for stages of few experts
    if (o.gemm_mode == MOE_GEMM_DENSE || o.pipeline_n != 1) return true;
    if (o.gemm_mode != MOE_GEMM_AUTO) return false;
    if (o.dense_min_rows > 0) return o.dense_min_rows <= d.tokens;
    return stage_experts(d, o) <= kAutoDenseMaxExperts;
}

// AUTO's choice for one stage of n experts with host row counts `rows`:
// DenseGemm (one launch per expert, tile height from its rows) when the
// launch-cost model predicts it faster than one grouped launch over the
// stage (or, with a fixed threshold m*, when every expert has >= m* rows).
bool auto_picks_dense(const moe_dims &d, const moe_opts &o, const int32_t *rows, int n, int grid,
                      bool split, double *group_us, double *dense_us) {
    int32_t max_rows = 0;
    for (int e = 0; e < n; ++e) max_rows = std::max(max_rows, rows[e]);
    const int bm_g = o.group_tile_rows > 0 ? o.group_tile_rows
                                           : group_launch_rows(max_rows, rows, n, 0, 0.0, d.hidden,
                                                               d.inter, grid, split);
    int64_t tiles_gu = 0, tiles_dn = 0;
    double dus = 0.0;
    int32_t min_rows = INT32_MAX;
    for (int e = 0; e < n; ++e) {
        tiles_gu += gemm_tiles(0, bm_g, rows[e], d.inter);
        tiles_dn += gemm_tiles(1, bm_g, rows[e], d.hidden);
        min_rows = std::min(min_rows, rows[e]);
        if (rows[e] > 0) {
            const int bm = o.dense_tile_rows > 0
                               ? o.dense_tile_rows
                               : dense_tile_rows(rows[e], d.hidden, d.inter, grid, split);
            dus += ffn_expert_us(bm, rows[e], d.hidden, d.inter, grid, split);
        }
    }
    const double gus = gemm_launch_us(0, bm_g, tiles_gu, d.hidden, grid, split) +
                       gemm_launch_us(1, bm_g, tiles_dn, d.inter, grid, split);
    if (group_us) *group_us = gus;
    if (dense_us) *dense_us = dus;
    if (o.dense_min_rows > 0) return min_rows >= o.dense_min_rows;
    if (n > kAutoDenseMaxExperts) return false;
    return dus < gus;
}

// ---- pipeline-number model (Sec. 5.2 items 4-5) ---------------------------
// On one GPU the communication of a stage is the stand-in for its two
// all2alls: the stage's combine (its gather is folded into the GEMM).  Its
// time comes from its bytes at the combine's measured streaming rate; the
// GEMM time of a stage from the launch-cost model of the GEMM kind AUTO
// would take for it.
constexpr double kCombineBytesPerUs = 5.6e6;  // ~5.6 TB/s, combine_kernel on MI355X
constexpr double kCombineLaunchUs = 4.0;
// Fixed cost of one more stage: the event hops between the GEMM and
// combine streams and the launches they separate.
constexpr double kStageUs = 20.0;
// The paper's thresholds for its DeepSeekV2 test (Sec. 5.2 item 4).
constexpr double kEps0Max = 0.32, kEps1Max = 0.03;
// The least predicted gain, as a fraction of the unsplit GEMM time, for
// which the library cuts stages: below it the gain is within the launch-cost
// model's error (4.5% rms per launch; measured, a predicted 7 us on the
// Zipf 4096-token load was a 57 us loss).
constexpr double kPnMinGainFrac = 0.05;

// A combine reads its stage's rows and every token's slot records; it
// writes every token's output when it starts y, and otherwise reads and
// writes only the tokens with a row in the stage (at most min(T, rows)).
double combine_us(const moe_dims &d, int64_t rows, bool accumulate) {
    const double touched = (double)std::min<int64_t>(d.tokens, rows);
    const double bytes = (double)rows * d.hidden * 4 +
                         (accumulate ? touched * d.hidden * 8 : (double)d.tokens * d.hidden * 4) +
                         (double)d.tokens * d.top_k * 8;
    return kCombineLaunchUs + bytes / kCombineBytesPerUs;
}

// GEMM and combine time of the expert stages of pipeline number n over the
// host row counts rows[0..EL).
void stage_times(const moe_dims &d, const moe_opts &o, const int32_t *rows, int n, int grid,
                 bool split, double *comm_us, double *comp_us) {
    const int EL = d.local_count, per = EL / n;
    double comm = 0.0, comp = 0.0;
    for (int i = 0; i < n; ++i) {
        const int32_t *r = rows + i * per;
        double gus = 0.0, dus = 0.0;
        const bool pick = auto_picks_dense(d, o, r, per, grid, split, &gus, &dus);
        const bool dense = o.gemm_mode == MOE_GEMM_DENSE || (o.gemm_mode == MOE_GEMM_AUTO && pick);
        comp += dense ? dus : gus;
        int64_t stage_rows = 0;
        for (int e = 0; e < per; ++e) stage_rows += r[e];
        comm += combine_us(d, stage_rows, d.shared_inter > 0 || i > 0);
    }
    *comm_us = comm;
    *comp_us = comp;
}

// The paper's terms for pipeline number n: T_comm and T_comp before the
// split, their sums over n stages (n S(m/n) and n G(m/n, E/n)), the
// enable-condition ratios and the gain L(n) - R(n).  The paper's
// L(n) = min(T_comm, T_comp) (n - 1) / n assumes the communication kernels
// run on SMs of their own beside the GEMM; on one GPU the persistent GEMM
// grid holds every CU it is given, so only the CUs it leaves free (a CU
// budget or side CUs) can run a combine beside it, and L is scaled by that
// fraction (none by default: measured, a combine next to a full-grid GEMM
// only runs in its tail).  R(n) is the overhead of cutting: the extra GEMM
// and combine time of n stages plus a fixed cost per added stage.
moe_pipeline_eval pipeline_eval(const moe_dims &d, const moe_opts &o, const int32_t *rows, int n,
                                int grid, bool split) {
    moe_pipeline_eval ev{};
    stage_times(d, o, rows, 1, grid, split, &ev.t_comm_us, &ev.t_comp_us);
    stage_times(d, o, rows, n, grid, split, &ev.t_comm_n_us, &ev.t_comp_n_us);
    ev.eps0 = ev.t_comm_us > 0 ? ev.t_comm_n_us / ev.t_comm_us - 1.0 : 0.0;
    ev.eps1 = ev.t_comp_us > 0 ? ev.t_comp_n_us / ev.t_comp_us - 1.0 : 0.0;
    const int cus = device_cu_count();
    ev.overlap_frac = cus > grid ? (double)(cus - grid) / cus : 0.0;
    const double C = std::min(ev.t_comm_us, ev.t_comp_us);
    const double R = (ev.t_comp_n_us - ev.t_comp_us) + (ev.t_comm_n_us - ev.t_comm_us) +
                     (n - 1) * kStageUs;
    ev.gain_us = n > 1 ? C * (n - 1) / n * ev.overlap_frac - R : 0.0;
    ev.enabled = (n == 1 || (ev.eps0 <= kEps0Max && ev.eps1 <= kEps1Max)) ? 1 : 0;
    return ev;
}

// pipeline_n = 0: the divisor of EL with the largest predicted gain among
// those that meet the enable condition, when that gain is at least
// kPnMinGainFrac of the unsplit GEMM time, else 1.
int choose_pipeline_auto(const moe_dims &d, const moe_opts &o, const int32_t *rows, int grid,
                         bool split) {
    int best = 1;
    double best_gain = 0.0;
    for (int n = 2; n <= d.local_count; ++n) {
        if (d.local_count % n) continue;
        const moe_pipeline_eval ev = pipeline_eval(d, o, rows, n, grid, split);
        if (ev.enabled && ev.gain_us > best_gain && ev.gain_us >= kPnMinGainFrac * ev.t_comp_us) {
            best = n;
            best_gain = ev.gain_us;
        }
    }
    return best;
}

int gemm_grid(const moe_opts &o) {
    int cus = device_cu_count();
    int grid = o.gemm_cu_budget > 0 ? o.gemm_cu_budget : cus;
    if (o.side_cus > 0) grid = std::min(grid, cus - o.side_cus);
    return std::max(8, (grid / 8) * 8);
}

// Scratch of the no-allocation entry point: one static buffer per device
// (each device holds its own copy of the array), reached through the address
// hipGetSymbolAddress gives for the current device.  Calls on one device
// share it, so they are serialised by g_noalloc_mu on the host; calls that
// overlap on the GPU (other streams, other processes do not share it) race.
__device__ __align__(256) char scratch[kNoAllocScratchBytes];
std::mutex g_noalloc_mu;
std::vector<char *> g_scratch_ptr;  // per device, under g_mu

moe_status noalloc_scratch(char **out) {
    int dev = 0;
    MOE_HIP(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lock(g_mu);
    if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize(dev + 1, nullptr);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        MOE_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(MOE_ERR_HIP, "hipGetSymbolAddress(scratch) gave NULL");
        g_scratch_ptr[dev] = static_cast<char *>(p);
    }
    *out = g_scratch_ptr[dev];
    return MOE_OK;
}

moe_status check_tensors(const moe_dims &d, const moe_bf16 *x, const float *w_router,
                         const moe_bf16 *w_gate, const moe_bf16 *w_up, const moe_bf16 *w_down,
                         const moe_bf16 *shared_gate, const moe_bf16 *shared_up,
                         const moe_bf16 *shared_down, const float *y) {
    if (!x || !w_router || !w_gate || !w_up || !w_down || !y)
        return fail(MOE_ERR_INVALID, "moe_ffn_forward: NULL tensor");
    if (d.shared_inter > 0 && (!shared_gate || !shared_up || !shared_down))
        return fail(MOE_ERR_INVALID, "moe_ffn_forward: shared_inter > 0 needs shared weights");
    return MOE_OK;
}

// The forward itself, after argument checks: workspace at `base` laid out
// as L.  st == NULL (the no-allocation entry point) runs every step on the
// caller's stream and never needs the row counts on the host.
// A roctx range over the host-side enqueue of one part of the forward (the
// whole call, the shared FFN, routing, dispatch, the wait for the row
// counts, each pipeline stage), shown by rocprofv3 --marker-trace beside the
// kernels; the calls cost next to nothing when no tool listens.
struct Marker {
    explicit Marker(const char *what) { roctxRangePushA(what); }
    ~Marker() { roctxRangePop(); }
    Marker(const Marker &) = delete;
    Marker &operator=(const Marker &) = delete;
};

moe_status forward_impl(const moe_dims &d, const moe_opts &opt, const moe_bf16 *x,
                        const float *w_router, const float *bias, const moe_bf16 *w_gate,
                        const moe_bf16 *w_up, const moe_bf16 *w_down,
                        const moe_bf16 *shared_gate, const moe_bf16 *shared_up,
                        const moe_bf16 *shared_down, float *y, int32_t *topk_ids, float *topk_w,
                        int32_t *counts, char *base, const WsLayout &L, DevState *st,
                        hipStream_t s0) {
    const moe_opts *o = &opt;
    const bool has_shared = d.shared_inter > 0;
    const bool tok_stages = o->chunk_mode == MOE_CHUNK_TOKENS;
    const int NB = L.nbuckets;

    int32_t *ids = topk_ids ? topk_ids : reinterpret_cast<int32_t *>(base + L.ids);
    float *wts = topk_w ? topk_w : reinterpret_cast<float *>(base + L.weights);
    // rows per bucket (local expert, or stage * EL + local expert) and their
    // prefix; the caller's counts are per local expert
    int32_t *cnt_el = counts ? counts
                             : reinterpret_cast<int32_t *>(base + (tok_stages ? L.counts_el
                                                                              : L.counts));
    int32_t *cnt = tok_stages ? reinterpret_cast<int32_t *>(base + L.counts) : cnt_el;
    int32_t *off = reinterpret_cast<int32_t *>(base + L.offsets);
    int32_t *sorted_slot = reinterpret_cast<int32_t *>(base + L.sorted_slot);
    int32_t *slot_row = reinterpret_cast<int32_t *>(base + L.slot_row);
    bf16_t *x_perm = reinterpret_cast<bf16_t *>(base + L.x_perm);
    bf16_t *act = reinterpret_cast<bf16_t *>(base + L.act);
    float *y_perm = reinterpret_cast<float *>(base + L.y_perm);
    bf16_t *shared_act = reinterpret_cast<bf16_t *>(base + L.shared_act);

    // pipeline number: given, or (0) chosen from the row counts below
    int PN = o->pipeline_n;
    const int EL = d.local_count;
    const int64_t tps = tok_stages ? (d.tokens + PN - 1) / PN : 0;
    // One stage without shared experts has nothing to overlap: every step
    // runs on the caller's stream (no cross-stream event hops, which cost
    // tens of microseconds each).  So does the serial mode, where nothing
    // may overlap, and the no-allocation entry point (no internal streams).
    // Otherwise gather, GEMMs and combine run on their own streams so that
    // stages (and the shared FFN) overlap.
    // (A library-chosen PN counts as pipelined here: the streams are set up
    // before the row counts are known.)
    const bool one_stream =
        st == nullptr || (PN == 1 && !has_shared) || (o->flags & MOE_FLAG_SERIAL) != 0;
    const int max_pn = PN > 0 ? PN : EL;
    hipEvent_t ev_fork = nullptr, ev_counts = nullptr, ev_done = nullptr, ev_start = nullptr;
    hipEvent_t ev_shared = nullptr;
    hipEvent_t *ev_g = nullptr, *ev_m = nullptr;
    Streams strm;
    if (st) {
        MOE_TRY(ensure_events(st->sync_ev, 3 * (size_t)max_pn + 5, hipEventDisableTiming));
        ev_fork = st->sync_ev[0];
        ev_counts = st->sync_ev[1];
        ev_done = st->sync_ev[2];
        ev_start = st->sync_ev[3];
        ev_shared = st->sync_ev[4];
        ev_g = &st->sync_ev[5];
        ev_m = ev_g + max_pn;
        if (!one_stream) MOE_TRY(get_streams(st, o->side_cus, &strm));
    }

    const bool timing = st && (o->flags & (MOE_FLAG_TIMING | MOE_FLAG_TIMING_GEMM)) != 0;
    std::vector<hipEvent_t> *tpool = nullptr;
    if (timing) {
        // a record that was read, or that holds another device's events,
        // starts anew; otherwise this call's spans are added to it
        int dev = 0;
        MOE_HIP(hipGetDevice(&dev));
        if ((int)t_time_ev.size() <= dev) t_time_ev.resize(dev + 1);
        tpool = &t_time_ev[dev];
        if (g_timing.read || g_timing.device != dev) {
            g_timing = TimingRecord{};
            g_timing.device = dev;
        }
        ++g_timing.calls;
    }
    Timer tm(tpool, timing ? o->flags : 0);
    hipStream_t sg = one_stream ? s0 : strm.sg;
    hipStream_t sm = one_stream ? s0 : strm.sm;
    hipStream_t sc = one_stream ? s0 : strm.sc;
    const int H = d.hidden, I = d.inter;
    const int64_t T = d.tokens;

    Marker mark_all("moe_ffn_forward");
    int total_span = -1;
    MOE_TRY(tm.begin(s0, PH_TOTAL, &total_span));
    // shared experts: independent of routing, start at once on the GEMM stream
    if (!one_stream) {
        MOE_HIP(hipEventRecord(ev_start, s0));
        MOE_HIP(hipStreamWaitEvent(sm, ev_start, 0));
        tm.gap();
    }
    // persistent grid of the grouped GEMMs (at most the CUs the GEMM stream
    // may use) and their K-split scratch (all on the GEMM stream, one GEMM
    // after another)
    const int grid = gemm_grid(*o);
    const bool split = (o->flags & MOE_FLAG_EXACT_ORDER) == 0;
    float *split_part = split ? reinterpret_cast<float *>(base + L.split_part) : nullptr;
    int32_t *split_meta = split ? reinterpret_cast<int32_t *>(base + L.split_meta) : nullptr;
    // the shared FFN's K split has scratch of its own when the workspace
    // holds it (then the routed GEMMs may run beside it)
    const bool shared_scratch = split && L.split_part_sh != 0;
    if (has_shared) {
        // the shared FFN is one expert of T contiguous rows through the
        // grouped scheduler, whose K split shortens a partial last round of
        // tiles (e.g. 1040 down tiles on 256 workgroups); same tile code, so
        // the same bits as a dense launch under MOE_FLAG_EXACT_ORDER
        Marker mark("moe shared FFN");
        moe_dims ds = d;
        ds.inter = d.shared_inter;
        ds.local_begin = 0;
        ds.local_count = 1;
        MOE_TRY(tm.begin(sm, PH_SHARED));
        // one expert of T rows, known on the host (no offsets array): the
        // height a dense launch of those rows takes
        const int bm_s = dense_tile_rows(T, H, d.shared_inter, grid, split);
        float *sp = shared_scratch ? reinterpret_cast<float *>(base + L.split_part_sh)
                                   : split_part;
        int32_t *sq = shared_scratch ? reinterpret_cast<int32_t *>(base + L.split_meta_sh)
                                     : split_meta;
        MOE_HIP(launch_group_gateup(ds, 0, 1, nullptr, x, nullptr, shared_gate, shared_up,
                                    shared_act, grid, sp, sq, bm_s, sm, T));
        MOE_HIP(launch_group_down(ds, 0, 1, nullptr, shared_act, shared_down, y, grid, sp, sq,
                                  bm_s, sm, T));
        MOE_TRY(tm.end(sm));
        if (!one_stream) MOE_HIP(hipEventRecord(ev_shared, sm));
    }

    // routing and dispatch indices on the caller stream
    {
        Marker mark("moe route");
        MOE_TRY(tm.begin(s0, PH_ROUTE));
        float *logits = L.logits ? reinterpret_cast<float *>(base + L.logits) : nullptr;
        MOE_HIP(launch_route(d, x, w_router, bias, ids, wts, logits, s0));
        MOE_TRY(tm.end(s0));
    }
    {
        Marker mark("moe dispatch");
        MOE_TRY(tm.begin(s0, PH_PERMUTE));
        MOE_HIP(launch_permute(d, ids, base, L, tps, cnt, off, cnt_el, sorted_slot, slot_row,
                               s0));
        MOE_TRY(tm.end(s0));
    }

    // GEMM kind per stage needs the row counts on the host
    std::vector<int32_t> hc;
    const bool need_counts = needs_host_counts(d, *o);
    if (need_counts) {
        if (!st) return fail(MOE_ERR_UNSUPPORTED, "row counts needed on the host");
        Marker mark("moe row counts to host");
        MOE_HIP(hipMemcpyAsync(st->pinned_counts, cnt, sizeof(int32_t) * NB,
                               hipMemcpyDeviceToHost, s0));
        MOE_HIP(hipEventRecord(ev_counts, s0));
        MOE_HIP(hipEventSynchronize(ev_counts));
        tm.gap();
        hc.assign(st->pinned_counts, st->pinned_counts + NB);
    }
    if (PN == 0) {
        PN = choose_pipeline_auto(d, *o, hc.data(), grid, split);
        if (timing) g_timing.pipeline_n = PN;
    } else if (timing) {
        g_timing.pipeline_n = PN;
    }
    const int per_stage = tok_stages ? EL : EL / PN;  // buckets per stage
    // the grouped gate/up GEMM can gather its token rows itself while every
    // byte offset into x fits 32 bits
    const bool fold_ok = gather_foldable(d);
    // Cross-stream hops cost host time (an event record or wait each) and
    // GPU latency, so only the ones that buy overlap are made: the gather
    // stream is used only when gathers run (not folded), and the combine
    // gets its own stream only when it can run beside a later stage's GEMMs;
    // with one stage it follows them on the GEMM stream.
    const bool combine_apart = !one_stream && PN > 1;
    // One stage beside the shared FFN: the routed GEMMs and the combine
    // follow the dispatch on the caller's stream (no hop to the GEMM stream
    // and back); only the combine, which adds onto the shared FFN's output,
    // waits for it.  This needs the shared FFN's own K-split scratch (the
    // two may overlap) and the folded gather (no gather stream).  Up to
    // kRoutedBesideSharedMaxTokens tokens: beyond, both GEMMs fill the chip
    // and running them side by side saves nothing (measured on the
    // DeepSeekV2 shape: -9% at 64 tokens, -4% at 4096, -0.7% at 16384,
    // where each GEMM then takes twice as long as alone).
    const bool routed_on_caller = !one_stream && PN == 1 && has_shared && fold_ok &&
                                  (!split || shared_scratch) &&
                                  T <= kRoutedBesideSharedMaxTokens;
    hipStream_t sr = routed_on_caller ? s0 : sm;  // the routed GEMMs' stream
    hipStream_t scomb = combine_apart ? sc : sr;

    if (!one_stream && !routed_on_caller) {
        MOE_HIP(hipEventRecord(ev_fork, s0));
        if (!fold_ok) MOE_HIP(hipStreamWaitEvent(sg, ev_fork, 0));
        MOE_HIP(hipStreamWaitEvent(sm, ev_fork, 0));
        if (combine_apart) MOE_HIP(hipStreamWaitEvent(sc, ev_fork, 0));
        tm.gap();
    }

    for (int i = 0; i < PN; ++i) {
        // buckets [b0, b0 + per_stage); their experts start at e_w (weights)
        const int b0 = i * per_stage;
        const int e_w = tok_stages ? 0 : b0;
        const int64_t t_lo = tok_stages ? std::min<int64_t>(T, i * tps) : 0;
        const int64_t t_hi = tok_stages ? std::min<int64_t>(T, (i + 1) * tps) : T;
        int64_t stage_rows = L.rcap;
        // rows of the stage's largest expert: the stage's tokens bound it,
        // the host counts give it exactly
        int64_t stage_max_rows = t_hi - t_lo;
        bool dense = o->gemm_mode == MOE_GEMM_DENSE;
        if (need_counts) {
            stage_rows = 0;
            stage_max_rows = 0;
            for (int b = b0; b < b0 + per_stage; ++b) {
                stage_rows += hc[b];
                stage_max_rows = std::max<int64_t>(stage_max_rows, hc[b]);
            }
            if (o->gemm_mode == MOE_GEMM_AUTO)
                dense = auto_picks_dense(d, *o, &hc[b0], per_stage, grid, split, nullptr,
                                         nullptr);
        }
        char stage_name[64];
        snprintf(stage_name, sizeof(stage_name), "moe stage %d of %d (%s)", i + 1, PN,
                 dense ? "dense" : "group");
        Marker mark(stage_name);
        // gather (dispatch of this stage), unless the gate/up GEMM reads its
        // token rows straight from x through sorted_slot
        const bool fold_gather = fold_ok;
        if (!fold_gather) {
            MOE_TRY(tm.begin(sg, PH_GATHER));
            MOE_HIP(launch_gather(d, b0, per_stage, off, sorted_slot, x, x_perm, stage_rows,
                                  sg));
            MOE_TRY(tm.end(sg));
        }
        if (!one_stream && !fold_gather) {
            MOE_HIP(hipEventRecord(ev_g[i], sg));
            MOE_HIP(hipStreamWaitEvent(sr, ev_g[i], 0));
            tm.gap();
        }

        // expert GEMMs; the grouped kernels index weights from their first
        // expert: the offsets are shifted so that expert e_w .. is bucket b0 ..
        const int32_t *goff = off + (b0 - e_w);
        const bf16_t *xrows = fold_gather ? x : x_perm;
        const int32_t *rmap = fold_gather ? sorted_slot : nullptr;
        if (dense) {
            // DenseGemm: one launch per expert, whose row count the host
            // knows, so each takes the tile height that fills the grid best
            if (timing) ++g_timing.dense_stages;
            for (int b = b0; b < b0 + per_stage; ++b) {
                const int64_t rows = hc[b];
                if (rows <= 0) continue;
                const int e = e_w + (b - b0);
                const int bm = o->dense_tile_rows > 0
                                   ? o->dense_tile_rows
                                   : dense_tile_rows(rows, H, I, grid, split);
                MOE_TRY(tm.begin(sr, PH_GATEUP));
                MOE_HIP(launch_group_gateup(d, e, 1, goff, xrows, rmap, w_gate, w_up, act, grid,
                                            split_part, split_meta, bm, sr));
                MOE_TRY(tm.end(sr));
                MOE_TRY(tm.begin(sr, PH_DOWN));
                MOE_HIP(launch_group_down(d, e, 1, goff, act, w_down, y_perm, grid, split_part,
                                          split_meta, bm, sr));
                MOE_TRY(tm.end(sr));
                if (timing) {
                    ++g_timing.gateup_launches;
                    ++g_timing.down_launches;
                }
            }
        } else {
            // GroupGemm: one launch over the stage's experts, row counts
            // read on the device
            if (timing) ++g_timing.group_stages;
            if (stage_rows > 0) {
                const int bm =
                    o->group_tile_rows > 0
                        ? o->group_tile_rows
                        : group_launch_rows(stage_max_rows, need_counts ? &hc[b0] : nullptr,
                                            per_stage, t_hi - t_lo, (double)d.top_k / d.experts,
                                            H, I, grid, split);
                MOE_TRY(tm.begin(sr, PH_GATEUP));
                MOE_HIP(launch_group_gateup(d, e_w, per_stage, goff, xrows, rmap, w_gate, w_up,
                                            act, grid, split_part, split_meta, bm, sr));
                MOE_TRY(tm.end(sr));
                // decode-sized stages with enough tiles: the skinny down tile
                const int64_t active =
                    std::min<int64_t>(per_stage, (t_hi - t_lo) * (int64_t)d.top_k);
                const int sk = skinny_down_rows(stage_max_rows, active, H);
                MOE_TRY(tm.begin(sr, PH_DOWN));
                if (sk > 0)
                    MOE_HIP(launch_skinny_down(d, e_w, per_stage, goff, act, w_down, y_perm, sk,
                                               active, sr));
                else
                    MOE_HIP(launch_group_down(d, e_w, per_stage, goff, act, w_down, y_perm, grid,
                                              split_part, split_meta, bm, sr));
                MOE_TRY(tm.end(sr));
                if (timing) {
                    ++g_timing.gateup_launches;
                    ++g_timing.down_launches;
                }
            }
        }
        if (combine_apart) {
            MOE_HIP(hipEventRecord(ev_m[i], sr));
            MOE_HIP(hipStreamWaitEvent(sc, ev_m[i], 0));
            tm.gap();
        }

        // weighted combine of this stage: its experts over all tokens, or
        // all experts over its tokens (after the shared FFN, onto its output)
        if (routed_on_caller) {
            MOE_HIP(hipStreamWaitEvent(s0, ev_shared, 0));
            tm.gap();
        }
        MOE_TRY(tm.begin(scomb, PH_COMBINE));
        const int accumulate = (has_shared || (!tok_stages && i > 0)) ? 1 : 0;
        MOE_HIP(launch_combine(d, tok_stages ? 0 : b0, tok_stages ? EL : per_stage, t_lo, t_hi,
                               y_perm, ids, slot_row, wts, y, accumulate, scomb));
        MOE_TRY(tm.end(scomb));
    }
    if (!one_stream && scomb != s0) {
        MOE_HIP(hipEventRecord(ev_done, scomb));
        MOE_HIP(hipStreamWaitEvent(s0, ev_done, 0));
        tm.gap();
    }
    MOE_TRY(tm.end(s0, total_span));
    if (timing) g_timing.valid = true;
    return MOE_OK;
}

}  // namespace moe

using namespace moe;

extern "C" {

moe_status moe_pipeline_plan(const moe_dims *dims, const moe_opts *opts, const int32_t *rows,
                             int32_t pipeline_n, moe_pipeline_eval *out) {
    MOE_TRY(check_dims(dims));
    moe_opts defaults{};
    defaults.pipeline_n = 1;
    const moe_opts *o = opts ? opts : &defaults;
    MOE_TRY(check_opts(dims, o));
    if (o->chunk_mode != MOE_CHUNK_EXPERTS)
        return fail(MOE_ERR_INVALID, "moe_pipeline_plan: expert stages only");
    if (!rows || !out) return fail(MOE_ERR_INVALID, "moe_pipeline_plan: NULL rows or out");
    const int EL = dims->local_count;
    for (int e = 0; e < EL; ++e)
        if (rows[e] < 0) return fail(MOE_ERR_INVALID, "moe_pipeline_plan: rows[%d] < 0", e);
    const int grid = gemm_grid(*o);
    const bool split = (o->flags & MOE_FLAG_EXACT_ORDER) == 0;
    int n = pipeline_n;
    if (n == 0) n = choose_pipeline_auto(*dims, *o, rows, grid, split);
    if (n < 1 || EL % n)
        return fail(MOE_ERR_INVALID, "moe_pipeline_plan: pipeline_n %d must divide %d",
                    pipeline_n, EL);
    *out = pipeline_eval(*dims, *o, rows, n, grid, split);
    out->pipeline_n = n;
    return MOE_OK;
}

moe_status moe_gemm_plan(const moe_dims *dims, const moe_opts *opts, int32_t n_experts,
                         const int32_t *rows, int32_t *dense, int32_t *tile_rows,
                         double *group_us, double *dense_us) {
    MOE_TRY(check_dims(dims));
    moe_opts defaults{};
    defaults.pipeline_n = 1;
    const moe_opts *o = opts ? opts : &defaults;
    MOE_TRY(check_opts(dims, o));
    if (n_experts < 1 || n_experts > kMaxExperts)
        return fail(MOE_ERR_INVALID, "moe_gemm_plan: n_experts %d outside [1, %d]", n_experts,
                    kMaxExperts);
    if (!rows || !dense) return fail(MOE_ERR_INVALID, "moe_gemm_plan: NULL rows or dense");
    for (int e = 0; e < n_experts; ++e)
        if (rows[e] < 0) return fail(MOE_ERR_INVALID, "moe_gemm_plan: rows[%d] < 0", e);
    const int grid = gemm_grid(*o);
    const bool split = (o->flags & MOE_FLAG_EXACT_ORDER) == 0;
    bool d_ = auto_picks_dense(*dims, *o, rows, n_experts, grid, split, group_us, dense_us);
    if (o->gemm_mode == MOE_GEMM_GROUP) d_ = false;
    if (o->gemm_mode == MOE_GEMM_DENSE) d_ = true;
    *dense = d_ ? 1 : 0;
    int32_t max_rows = 0;
    for (int e = 0; e < n_experts; ++e) max_rows = std::max(max_rows, rows[e]);
    if (tile_rows)
        for (int e = 0; e < n_experts; ++e)
            tile_rows[e] = !d_ ? (o->group_tile_rows > 0
                                      ? o->group_tile_rows
                                      : group_launch_rows(max_rows, rows, n_experts, 0, 0.0,
                                                          dims->hidden, dims->inter, grid, split))
                           : rows[e] == 0 ? 0
                           : o->dense_tile_rows > 0
                               ? o->dense_tile_rows
                               : dense_tile_rows(rows[e], dims->hidden, dims->inter, grid, split);
    return MOE_OK;
}

// The pipeline-number model of the paper's ablation (Sec. 5.2): the overlap
// hides C/PN of each of PN - 1 stages, and cutting the work costs
// k*PN + b, so G(PN) = C - b - (C/PN + k*PN) for PN > 1 and G(1) = 0.  The
// candidates are the divisors of local_count (each stage an equal expert
// group), searched exhaustively: the closed-form optimum sqrt(C/k) need not
// be one of them.
moe_status moe_choose_pipeline_n(double c_ms, double k_ms, double b_ms, int32_t local_count,
                                 int32_t *pn, double *gain_ms) {
    if (!pn) return fail(MOE_ERR_INVALID, "moe_choose_pipeline_n: NULL pn");
    if (!std::isfinite(c_ms) || !std::isfinite(k_ms) || !std::isfinite(b_ms) || c_ms < 0 ||
        k_ms < 0)
        return fail(MOE_ERR_INVALID, "moe_choose_pipeline_n: C and k must be finite and >= 0, "
                                     "b finite");
    if (local_count < 1 || local_count > kMaxExperts)
        return fail(MOE_ERR_INVALID, "moe_choose_pipeline_n: local_count %d out of range",
                    local_count);
    int32_t best = 1;
    double best_gain = 0.0;
    for (int32_t n = 2; n <= local_count; ++n) {
        if (local_count % n) continue;
        const double g = c_ms - b_ms - (c_ms / n + k_ms * n);
        if (g > best_gain) {
            best = n;
            best_gain = g;
        }
    }
    *pn = best;
    if (gain_ms) *gain_ms = best_gain;
    return MOE_OK;
}

moe_status moe_ffn_forward(const moe_dims *dims, const moe_opts *opts, const moe_bf16 *x,
                           const float *w_router, const float *bias,
                           const moe_bf16 *w_gate, const moe_bf16 *w_up,
                           const moe_bf16 *w_down, const moe_bf16 *shared_gate,
                           const moe_bf16 *shared_up, const moe_bf16 *shared_down,
                           float *y, int32_t *topk_ids, float *topk_w, int32_t *counts,
                           void *ws, size_t ws_bytes, void *stream) {
    MOE_TRY(check_dims(dims));
    moe_opts defaults{};
    defaults.pipeline_n = 1;
    const moe_opts *o = opts ? opts : &defaults;
    MOE_TRY(check_opts(dims, o));
    if (dims->tokens == 0) return MOE_OK;
    MOE_TRY(check_tensors(*dims, x, w_router, w_gate, w_up, w_down, shared_gate, shared_up,
                          shared_down, y));
    const WsLayout L = ws_layout(dims, o);
    if (!ws || ws_bytes < L.total)
        return fail(MOE_ERR_WORKSPACE, "moe_ffn_forward: workspace %zu < %zu bytes", ws_bytes,
                    L.total);
    DevState *st = nullptr;
    MOE_TRY(get_state(&st));
    std::lock_guard<std::mutex> call(st->call);
    return forward_impl(*dims, *o, x, w_router, bias, w_gate, w_up, w_down, shared_gate,
                        shared_up, shared_down, y, topk_ids, topk_w, counts,
                        static_cast<char *>(ws), L, st, (hipStream_t)stream);
}

moe_status moe_ffn_forward_noalloc(const moe_dims *dims, const moe_opts *opts,
                                   const moe_bf16 *x, const float *w_router, const float *bias,
                                   const moe_bf16 *w_gate, const moe_bf16 *w_up,
                                   const moe_bf16 *w_down, const moe_bf16 *shared_gate,
                                   const moe_bf16 *shared_up, const moe_bf16 *shared_down,
                                   float *y, int32_t *topk_ids, float *topk_w, int32_t *counts,
                                   void *stream) {
    MOE_TRY(check_dims(dims));
    moe_opts defaults{};
    defaults.pipeline_n = 1;
    const moe_opts *o = opts ? opts : &defaults;
    MOE_TRY(check_opts(dims, o));
    if (o->flags & (MOE_FLAG_TIMING | MOE_FLAG_TIMING_GEMM))
        return fail(MOE_ERR_UNSUPPORTED, "moe_ffn_forward_noalloc: no timing flags");
    if (needs_host_counts(*dims, *o))
        return fail(MOE_ERR_UNSUPPORTED,
                    "moe_ffn_forward_noalloc: options need the row counts on the host "
                    "(pipeline_n > 1, DenseGemm, or an AUTO threshold within reach)");
    if (dims->tokens == 0) return MOE_OK;
    MOE_TRY(check_tensors(*dims, x, w_router, w_gate, w_up, w_down, shared_gate, shared_up,
                          shared_down, y));
    const WsLayout L = ws_layout(dims, o, false);
    if (L.total > kNoAllocScratchBytes)
        return fail(MOE_ERR_UNSUPPORTED,
                    "moe_ffn_forward_noalloc: needs %zu bytes of scratch, the built-in "
                    "buffer holds %zu",
                    L.total, kNoAllocScratchBytes);
    char *base = nullptr;
    MOE_TRY(noalloc_scratch(&base));
    std::lock_guard<std::mutex> call(g_noalloc_mu);
    return forward_impl(*dims, *o, x, w_router, bias, w_gate, w_up, w_down, shared_gate,
                        shared_up, shared_down, y, topk_ids, topk_w, counts, base, L, nullptr,
                        (hipStream_t)stream);
}

moe_status moe_last_timing(moe_timing *out) {
    if (!out) return fail(MOE_ERR_INVALID, "moe_last_timing: NULL");
    if (!g_timing.valid) return fail(MOE_ERR_INVALID, "moe_last_timing: no timed call");
    float ph[PH_N] = {0};
    for (const TimedSpan &sp : g_timing.spans) {
        MOE_HIP(hipEventSynchronize(sp.stop));
        float ms = 0.f;
        MOE_HIP(hipEventElapsedTime(&ms, sp.start, sp.stop));
        ph[sp.phase] += ms;
    }
    *out = moe_timing{};
    out->route_ms = ph[PH_ROUTE];
    out->permute_ms = ph[PH_PERMUTE];
    out->gather_ms = ph[PH_GATHER];
    out->gateup_ms = ph[PH_GATEUP];
    out->down_ms = ph[PH_DOWN];
    out->shared_ms = ph[PH_SHARED];
    out->combine_ms = ph[PH_COMBINE];
    out->total_ms = ph[PH_TOTAL];
    out->gateup_launches = g_timing.gateup_launches;
    out->down_launches = g_timing.down_launches;
    out->dense_stages = g_timing.dense_stages;
    out->group_stages = g_timing.group_stages;
    out->pipeline_n = g_timing.pipeline_n;
    out->calls = g_timing.calls;
    g_timing.read = true;
    return MOE_OK;
}

}  // extern "C"
