/*
 * moe.h -- C ABI of the MI355X (gfx950) routed MoE FFN forward, the hot path
 * of EPS-MoE (arXiv 2410.12247): top-k softmax gating, expert-sorted
 * dispatch, the SwiGLU expert FFN run as one grouped GEMM or as per-expert
 * dense GEMMs, and the weighted combine, for one GPU's share of experts.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensor pointers are DEVICE pointers owned by the caller; the library
 *   never frees or retains them.  moe_dims and moe_opts live in host memory.
 * - Layouts are row-major and dense.  bf16 tensors are passed as their
 *   16-bit patterns (moe_bf16).  Expert weights use the [out, in] layout of
 *   a linear layer, so both GEMM operands are contiguous along the reduced
 *   dimension:  w_gate, w_up [EL][I][H];  w_down [EL][H][I];  shared
 *   gate/up [Is][H], shared down [H][Is].
 * - Every call is asynchronous on `stream` (a hipStream_t; NULL is the null
 *   stream) unless stated otherwise.
 * - Arguments are checked on the host before anything is enqueued; a bad
 *   argument returns MOE_ERR_INVALID / MOE_ERR_UNSUPPORTED /
 *   MOE_ERR_WORKSPACE and leaves every buffer untouched.  A failing HIP call
 *   returns MOE_ERR_HIP.  moe_last_error() gives the message of the last
 *   failure on the calling thread.  Nothing aborts or throws.
 * - tokens == 0 is a valid no-op.
 * - Supported sizes: 1 <= experts <= 256, 1 <= top_k <= min(experts, 8),
 *   hidden, inter and shared_inter multiples of 64, local experts
 *   [local_begin, local_begin + local_count) inside [0, experts),
 *   tokens * top_k < 2^31.
 * - Results are deterministic: the same inputs and options give the same
 *   bits on every run.  With MOE_FLAG_EXACT_ORDER (and in moe_ffn_group and
 *   moe_ffn_dense) every expert-GEMM output is one pass over K, so the bits
 *   are also the same for any pipeline number, stage kind, CU budget and
 *   either GEMM kind.  Without it the grouped GEMM may cut the tiles of its
 *   last, partial round into K pieces summed in a fixed order, which moves
 *   the last bits of those outputs with the launch's tile count.
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t moe_bf16; /* bf16 bit pattern */

typedef enum {
    MOE_OK = 0,
    MOE_ERR_INVALID = 1,     /* null pointer, size out of range, bad option */
    MOE_ERR_UNSUPPORTED = 2, /* experts > 256 or top_k > 8 */
    MOE_ERR_WORKSPACE = 3,   /* workspace smaller than moe_workspace_bytes() */
    MOE_ERR_HIP = 4          /* a HIP runtime call failed */
} moe_status;

/* Problem shape.  T tokens of width H are routed over E experts (top-k);
 * this GPU computes local experts [local_begin, local_begin + local_count),
 * each a SwiGLU FFN of width I, plus optional shared experts applied to
 * every token whose concatenated width is shared_inter (0 = none). */
typedef struct {
    int64_t tokens;       /* T */
    int32_t hidden;       /* H */
    int32_t inter;        /* I */
    int32_t experts;      /* E, router width */
    int32_t top_k;        /* k */
    int32_t local_begin;  /* e0 */
    int32_t local_count;  /* EL */
    int32_t renormalize;  /* 1: softmax over the k selected; 0: over all E */
    int32_t shared_inter; /* Is (0 = no shared experts) */
} moe_dims;

enum { MOE_GEMM_AUTO = 0, MOE_GEMM_GROUP = 1, MOE_GEMM_DENSE = 2 };
enum { MOE_CHUNK_EXPERTS = 0, MOE_CHUNK_TOKENS = 1 };
enum {
    MOE_FLAG_TIMING = 1,
    MOE_FLAG_TIMING_GEMM = 2,
    MOE_FLAG_EXACT_ORDER = 4,
    MOE_FLAG_SERIAL = 8
};

/* Options of moe_ffn_forward (Sec. 4.3 of the paper: the GroupGemm /
 * DenseGemm switch by load, the pipeline number PN and how the work is cut
 * into pipeline stages).
 * chunk_mode MOE_CHUNK_EXPERTS (default): stage s is the expert group
 *   [s*EL/PN, (s+1)*EL/PN) with all of its rows, so each expert's weights
 *   are read by one stage only (the paper's horizontal split with weights
 *   split by expert, Sec. 4.3).  PN must divide local_count.
 * chunk_mode MOE_CHUNK_TOKENS: stage s is the token range
 *   [s*ceil(T/PN), (s+1)*ceil(T/PN)) over all local experts, so every stage
 *   reads every local expert's weights again (the split the paper argues
 *   against); kept as a measured comparison.  Needs PN*local_count <= 256.
 * Both modes give the same bits under MOE_FLAG_EXACT_ORDER. */
typedef struct {
    int32_t gemm_mode;      /* MOE_GEMM_AUTO, _GROUP or _DENSE */
    int32_t dense_min_rows; /* 0: AUTO weighs GroupGemm against DenseGemm
                               for each stage of at most two experts with
                               the library's launch-cost model (see
                               moe_gemm_plan) and takes GroupGemm for larger
                               stages.  > 0: AUTO picks DenseGemm for a
                               stage when every expert in it has at least
                               this many rows (Sec. 3.2 Conclusion 1's
                               threshold m), else GroupGemm */
    int32_t pipeline_n;     /* PN >= 1, the number of pipeline stages; 0 = chosen
                               by the library from the row counts (expert
                               stages only; see moe_pipeline_plan) */
    int32_t gemm_cu_budget; /* workgroups of the persistent grouped GEMM;
                               0 = one per compute unit */
    int32_t flags;          /* MOE_FLAG_TIMING: time each phase with HIP
                               events (read with moe_last_timing).
                               MOE_FLAG_TIMING_GEMM: time only the expert
                               GEMM launches (gate/up, down, shared), with
                               one event between consecutive launches of a
                               stream; the other phases read 0.  Every
                               event recorded between two kernels delays
                               the second, so this is the mode to time a
                               run whose wall time also matters.
                               MOE_FLAG_EXACT_ORDER: no K split in the
                               grouped GEMM (see the determinism note at
                               the top); slower when the tile count leaves
                               a partial last round of the grid.
                               MOE_FLAG_SERIAL: every step of every stage
                               (and the shared experts) runs on the caller's
                               stream in order, so nothing overlaps: the
                               paper's serial mode (Sec. 5.2), which
                               measures what cutting the work into PN stages
                               costs by itself.  Same bits as without it. */
    int32_t chunk_mode;     /* MOE_CHUNK_EXPERTS or MOE_CHUNK_TOKENS */
    int32_t dense_tile_rows;/* token rows of a DenseGemm tile: 0 = chosen per
                               expert from its row count (the height whose
                               tile count fills the chip best), or 128, 192,
                               256, 320 to force one */
    int32_t side_cus;       /* Sec. 5.2's SM control: when the forward uses
                               its side streams (PN != 1 or shared experts),
                               0 = no CU masks; > 0 = the gather and combine
                               streams run on this many CUs (spread over the
                               XCDs) and the GEMM stream, with its persistent
                               grid, on the others.  At most 248. */
    int32_t group_tile_rows;/* token rows of a GroupGemm tile: 0 = chosen per
                               stage by the launch-cost model (never taller
                               than the smallest height that holds the
                               stage's largest expert), or 128, 192, 256,
                               320 to force one */
} moe_opts;

/* Per-phase device time, in milliseconds summed over stages and over the
 * timed moe_ffn_forward calls (MOE_FLAG_TIMING or MOE_FLAG_TIMING_GEMM) this
 * thread made on one device since it last called moe_last_timing (`calls`
 * of them), so a timed loop needs one read at its end, not a host sync per
 * step.  Launch and stage counts add up the same way; pipeline_n is the
 * last call's. */
typedef struct {
    float route_ms, permute_ms, gather_ms, gateup_ms, down_ms, shared_ms,
        combine_ms, total_ms;
    int32_t gateup_launches, down_launches; /* GEMM kernel launches timed */
    int32_t dense_stages, group_stages;     /* policy decisions taken */
    int32_t pipeline_n;                     /* stages the last call ran */
    int32_t calls;                          /* timed calls summed */
} moe_timing;

/* The paper's pipeline-number analysis (Sec. 5.2 items 4-5) for one
 * forward, evaluated with the library's cost models. */
typedef struct {
    double t_comm_us;   /* T_comm before the split: the combine, one-GPU
                           stand-in for the dispatch and combine all2alls */
    double t_comp_us;   /* T_comp before the split: the expert GEMMs */
    double t_comm_n_us; /* N * S(m/N): the stages' combines, summed */
    double t_comp_n_us; /* N * G(m/N, E/N): the stages' GEMMs, summed */
    double eps0;        /* N * S(m/N) / S(m) - 1 */
    double eps1;        /* N * G(m/N, E/N) / G(m, E) - 1 */
    double overlap_frac;/* share of the CUs the GEMM grid leaves free for
                           the side streams (CU budget or side_cus): the
                           part of L(N) one GPU can realise */
    double gain_us;     /* L(N) - R(N): min(T_comm, T_comp) (N - 1) / N *
                           overlap_frac, minus the split's extra GEMM and
                           combine time and a fixed cost per added stage */
    int32_t enabled;    /* eps0 <= 0.32 and eps1 <= 0.03 (the values of the
                           paper's DeepSeekV2 test), or N = 1 */
    int32_t pipeline_n; /* N */
} moe_pipeline_eval;

/* Bytes of device workspace: with opts == NULL, what moe_permute needs;
 * with opts != NULL, what moe_ffn_forward needs with those options (a
 * superset).  Host-only; never touches the GPU.  Returns 0 for invalid dims
 * or options. */
size_t moe_workspace_bytes(const moe_dims *dims, const moe_opts *opts);

/* Guard gaps of the workspace layout (a debugging aid for out-of-region
 * writes; no passage of the paper defines it).  After every region of the
 * layout moe_workspace_bytes() sizes, the library leaves MOE_WS_GUARD_BYTES
 * bytes that no call reads or writes: a caller may fill them with a canary
 * before a call and compare them after it.  Writes the byte offsets of the
 * first `capacity` gaps (from the workspace start) to `offsets` and returns
 * how many gaps the layout has; -1 for invalid dims or options, or for
 * offsets == NULL with capacity > 0.  opts as in moe_workspace_bytes.
 * Host-only; never touches the GPU. */
#define MOE_WS_GUARD_BYTES 256
int32_t moe_workspace_guards(const moe_dims *dims, const moe_opts *opts, int64_t *offsets,
                             int32_t capacity);

/* Router (the topKGating operator of Sec. 3.3; k of E experts per token as
 * in Sec. 3.2).  For each token t:
 *   z[e] = fp32 fused-multiply-add chain over h = 0..H-1 (ascending, from
 *          +0) of x[t][h] * w_router[e][h], then + bias[e] (one fp32 add)
 *   topk_ids[t][0..k)  the k largest z, by (z descending, e ascending);
 *                      -0 and +0 are equal
 *   topk_w[t][j]       softmax weight, computed in fp64 and rounded to fp32:
 *                      over the k selected logits when renormalize, else
 *                      over all E logits.
 * x [T][H] bf16; w_router [E][H] fp32; bias [E] fp32 or NULL;
 * topk_ids [T][k] int32 (global expert ids); topk_w [T][k] fp32.
 * Logits are never materialised.  NaN logits are not supported. */
moe_status moe_route(const moe_dims *dims, const moe_bf16 *x, const float *w_router,
                     const float *bias, int32_t *topk_ids, float *topk_w, void *stream);

/* Dispatch (Fig. 7a: each expert takes its tokens in ascending order;
 * Sec. 4.3: inputs split by rows, weights by expert).  Rows are ordered by
 * (local expert ascending, token ascending):
 *   counts [EL]        rows of each local expert
 *   offsets [EL+1]     exclusive prefix of counts (unpadded)
 *   sorted_slot [R]    row -> slot t*k+j   (R = offsets[EL] <= T*min(k,EL);
 *                      the buffer must hold T*min(k,EL) entries)
 *   slot_row [T*k]     slot -> row, -1 when the slot's expert is not local
 *   x_perm [R][H]      x_perm[r] = x[sorted_slot[r] / k]; may be NULL to
 *                      build the indices only (then x may be NULL too)
 * Deterministic: scan-based, no atomics decide an order.
 * ws: device workspace of at least moe_workspace_bytes(dims, NULL) bytes. */
moe_status moe_permute(const moe_dims *dims, const int32_t *topk_ids, const moe_bf16 *x,
                       int32_t *counts, int32_t *offsets, int32_t *sorted_slot,
                       int32_t *slot_row, moe_bf16 *x_perm, void *ws, size_t ws_bytes,
                       void *stream);

/* Gather of the rows of local experts [e_first, e_first + e_count) only:
 * x_perm[r] = x[sorted_slot[r] / k] for r in [offsets[e_first],
 * offsets[e_first + e_count]).  offsets and sorted_slot are device arrays
 * from moe_permute.  The dispatch of one pipeline stage. */
moe_status moe_gather(const moe_dims *dims, int32_t e_first, int32_t e_count,
                      const int32_t *offsets, const int32_t *sorted_slot,
                      const moe_bf16 *x, moe_bf16 *x_perm, void *stream);

/* GroupGemm expert FFN (Sec. 3.2, Conclusions 1-3; Fig. 3): ONE launch per
 * GEMM for all rows of local experts [e_first, e_first + e_count), each
 * expert with its own row count read on the device from offsets, so no
 * host synchronisation is needed.  For every such row r of expert e:
 *   act[r]    = bf16( silu(g) * u ), g = w_gate[e] x_perm[r],
 *                                     u = w_up[e] x_perm[r]   (fp32 accum)
 *   y_perm[r] = w_down[e] act[r]                               (fp32 accum)
 * bf16 MFMA with fp32 accumulation; silu(g) = g / (1 + exp(-g)).
 * w_gate/w_up/w_down point at the stacks of all EL local experts.
 * act [R][I] bf16 (caller scratch, rows indexed like x_perm);
 * y_perm [R][H] fp32.  cu_budget: persistent grid size (0 = all CUs).
 * Takes no workspace, so every tile is one pass over K (the bits of
 * moe_ffn_forward with MOE_FLAG_EXACT_ORDER). */
moe_status moe_ffn_group(const moe_dims *dims, int32_t e_first, int32_t e_count,
                         const int32_t *offsets, const moe_bf16 *x_perm,
                         const moe_bf16 *w_gate, const moe_bf16 *w_up,
                         const moe_bf16 *w_down, moe_bf16 *act, float *y_perm,
                         int32_t cu_budget, void *stream);

/* DenseGemm expert FFN (Sec. 4.3: with one expert per pipeline stage the
 * grouped GEMM becomes a dense one): one dense SwiGLU FFN over `rows`
 * contiguous rows whose count is known on the host, so the launch takes the
 * tile height (128 to 320 token rows) whose tile count fills the chip best:
 *   act[r] = bf16(silu(w_gate x[r]) * (w_up x[r])),  y[r] = w_down act[r]
 * x [rows][hidden] bf16; w_gate, w_up [inter][hidden]; w_down
 * [hidden][inter]; act [rows][inter] bf16 scratch; y [rows][hidden] fp32.
 * Usable for shared experts (inter = shared width, x = all tokens), which
 * moe_ffn_forward runs through the grouped scheduler instead (one expert
 * of T rows).  Same arithmetic and bits as moe_ffn_group for the same
 * rows. */
moe_status moe_ffn_dense(int64_t rows, int32_t hidden, int32_t inter, const moe_bf16 *x,
                         const moe_bf16 *w_gate, const moe_bf16 *w_up,
                         const moe_bf16 *w_down, moe_bf16 *act, float *y, void *stream);

/* Combine (LocalReduce, Fig. 7b) of the local experts [e_first,
 * e_first + e_count):  for every token t,
 *   y[t] = (accumulate ? y[t] : 0) + sum_j topk_w[t][j] * y_perm[slot_row[t*k+j]]
 * over the slots j whose expert lies in that range, the terms taken in
 * ascending expert order, each added with one fp32 fused multiply-add.
 * Running the stages of a pipeline in order (first with accumulate = 0, or
 * all with accumulate = 1 over a y that holds the shared experts' output)
 * gives the same bits as one call over all local experts.
 * y_perm [R][H] fp32; topk_ids, slot_row [T][k] int32; topk_w [T][k];
 * y [T][H] fp32. */
moe_status moe_combine(const moe_dims *dims, int32_t e_first, int32_t e_count,
                       const float *y_perm, const int32_t *topk_ids, const int32_t *slot_row,
                       const float *topk_w, float *y, int32_t accumulate, void *stream);

/* The whole forward of one MoE layer's routed FFN for this GPU's experts:
 * route -> dispatch -> per pipeline stage { gather ; GroupGemm or DenseGemm
 * (picked per stage from its row counts, Sec. 3.2 Conclusion 1 and
 * Sec. 4.3) ; combine }, with stage i+1's gather and stage i-1's combine
 * running on their own streams beside stage i's GEMMs (the one-GPU form of
 * the expert pipeline of Sec. 4.3-4.4).  The shared experts (if any) run
 * first, as one grouped-GEMM expert of all T rows, and write y; otherwise
 * the first combine writes every token.
 * topk_ids, topk_w, counts: optional outputs (NULL = keep them in the
 * workspace).  shared_*: required iff dims->shared_inter > 0.
 * ws: at least moe_workspace_bytes(dims, opts) bytes of device memory.
 * Ordered after prior work on `stream` and finished on `stream`.  When the
 * policy needs row counts on the host (gemm_mode != GROUP or PN > 1) the
 * call blocks the host once on a 4*EL-byte device-to-host copy (AUTO needs
 * the counts only when its threshold can be reached by some expert).
 * Thread safety: calls from several host threads on one device are
 * serialised inside the library (the side streams, ordering events and the
 * pinned copy of the counts are per device); moe_last_timing reads the
 * calling thread's own timed calls. */
moe_status moe_ffn_forward(const moe_dims *dims, const moe_opts *opts, const moe_bf16 *x,
                           const float *w_router, const float *bias,
                           const moe_bf16 *w_gate, const moe_bf16 *w_up,
                           const moe_bf16 *w_down, const moe_bf16 *shared_gate,
                           const moe_bf16 *shared_up, const moe_bf16 *shared_down,
                           float *y, int32_t *topk_ids, float *topk_w, int32_t *counts,
                           void *ws, size_t ws_bytes, void *stream);

/* moe_ffn_forward for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, arguments and bits as moe_ffn_forward with the same
 * options, but it takes no workspace.  Its scratch is a static device buffer
 * of 256 MiB in the library (each device the library runs on holds its own
 * copy until the process ends); the call allocates nothing, on the device or
 * the host.  Limits: moe_workspace_bytes(dims, opts) must not exceed
 * 256 MiB (e.g. up to 512 tokens of the Mixtral-, DBRX- and DeepSeekV2-shaped
 * layers, or decode batches), else MOE_ERR_UNSUPPORTED; options that need
 * the row counts on the host (pipeline_n > 1, MOE_GEMM_DENSE, or an AUTO
 * threshold some expert can reach) and the timing flags are refused with
 * MOE_ERR_UNSUPPORTED; every step runs on `stream` (shared experts
 * included), with the same bits as with side streams.  All calls on one
 * device share the buffer, and it keeps the last call's contents: calls from
 * several host threads are serialised, but calls that overlap on the GPU
 * (this one still running when another is enqueued on another stream) race
 * on it.  Nothing in the buffer needs to start zeroed. */
moe_status moe_ffn_forward_noalloc(const moe_dims *dims, const moe_opts *opts,
                                   const moe_bf16 *x, const float *w_router, const float *bias,
                                   const moe_bf16 *w_gate, const moe_bf16 *w_up,
                                   const moe_bf16 *w_down, const moe_bf16 *shared_gate,
                                   const moe_bf16 *shared_up, const moe_bf16 *shared_down,
                                   float *y, int32_t *topk_ids, float *topk_w, int32_t *counts,
                                   void *stream);

/* Timing of the timed moe_ffn_forward calls on this thread since the
 * previous read (waits for their events); the next timed call then starts a
 * new record.  Returns MOE_ERR_INVALID when no timed call was made. */
moe_status moe_last_timing(moe_timing *out);

/* The paper's enable condition and gain for PN = pipeline_n expert stages
 * (pipeline_n = 0: the PN moe_ffn_forward would choose with pipeline_n = 0,
 * i.e. the divisor of local_count with the largest gain among those
 * enabled, when that gain is at least 5% of the unsplit GEMM time (the
 * launch-cost model's error), else 1), from the host row counts
 * rows[0..local_count) of the local experts.  The GEMM terms use the launch-cost model of the GEMM
 * kind AUTO (or opts->gemm_mode) takes per stage; the communication terms
 * the combine's bytes at its measured streaming rate.  Expert stages only.
 * Host-only; never touches the GPU. */
moe_status moe_pipeline_plan(const moe_dims *dims, const moe_opts *opts, const int32_t *rows,
                             int32_t pipeline_n, moe_pipeline_eval *out);

/* The GEMM plan AUTO makes for one pipeline stage (Sec. 3.2 Conclusion 1:
 * GroupGemm and DenseGemm each win over part of the load range; Sec. 4.3:
 * with one expert per stage the grouped GEMM becomes a dense one), from the
 * host row counts of its n_experts experts, rows[0..n_experts).  The model
 * prices each launch from measured per-tile costs of every tile height:
 * GroupGemm is one launch over the stage with one tile height (the model's
 * cheapest up to the smallest height that holds the largest expert, taken
 * when at least 5% below that height's price; or opts->group_tile_rows);
 * DenseGemm is one launch per expert with its own tile height.  Writes *dense (1 when
 * the stage would run DenseGemm under opts->gemm_mode, AUTO included) and,
 * when not NULL, tile_rows[e] (the tile height of expert e's launch, 0 for
 * an empty expert), *group_us and *dense_us (predicted GEMM microseconds
 * of the two kinds).  Uses dims->hidden / inter, opts->gemm_cu_budget,
 * dense_min_rows, dense_tile_rows, group_tile_rows and MOE_FLAG_EXACT_ORDER.  Host-only;
 * never touches the GPU (the grid is the current device's CU count, 256
 * when no device is visible). */
moe_status moe_gemm_plan(const moe_dims *dims, const moe_opts *opts, int32_t n_experts,
                         const int32_t *rows, int32_t *dense, int32_t *tile_rows,
                         double *group_us, double *dense_us);

/* Pipeline number from the overhead model of the paper's ablation (Sec. 5.2):
 * PN stages hide (PN - 1)/PN of C = min(T_comm, T_comp), the smaller of the
 * unsplit communication and computation times, and cost R(PN) = k*PN + b, so
 * the latency gain of PN > 1 is G(PN) = C - b - (C/PN + k*PN), largest near
 * PN = sqrt(C/k).  Writes to *pn the PN in [1, local_count] that divides
 * local_count and maximises G, with G(1) = 0 (no pipeline, no overhead); a
 * pipeline is chosen only when its gain is positive, and ties go to the
 * smaller PN.  k = 0 (no per-stage overhead) picks the largest PN whose gain
 * is positive.  *gain_ms (may be NULL) receives G(*pn).  Times in ms; c_ms
 * and k_ms must be finite and >= 0, b_ms finite, local_count in [1, 256],
 * else MOE_ERR_INVALID.  Host-only; never touches the GPU. */
moe_status moe_choose_pipeline_n(double c_ms, double k_ms, double b_ms, int32_t local_count,
                                 int32_t *pn, double *gain_ms);

const char *moe_status_string(moe_status s);
const char *moe_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* MOE_H */
