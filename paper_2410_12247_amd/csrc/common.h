// Internal declarations shared by the HIP sources of libmoe.so.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "moe.h"

namespace moe {

using bf16_t = uint16_t;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxExperts = 256;
constexpr int kMaxTopK = 8;
constexpr int kDimAlign = 64;  // hidden / inter multiple

// Records `msg` as the calling thread's last error and returns `s`.
moe_status fail(moe_status s, const char *fmt, ...);
// Checks a HIP return code; on failure records it and returns MOE_ERR_HIP.
moe_status hip_check(hipError_t e, const char *what);

#define MOE_HIP(expr)                                              \
    do {                                                           \
        moe_status _s = ::moe::hip_check((expr), #expr);           \
        if (_s != MOE_OK) return _s;                               \
    } while (0)

#define MOE_TRY(expr)                      \
    do {                                   \
        moe_status _s = (expr);            \
        if (_s != MOE_OK) return _s;       \
    } while (0)

// Host-side validation of the dims every entry point uses.
moe_status check_dims(const moe_dims *d);

// Number of compute units of the current device (cached per device).
int device_cu_count();

// Workspace layout used by moe_permute and moe_ffn_forward.  The dispatch
// orders rows by a bucket index: the local expert (EXPERTS stages) or
// token-range stage * EL + local expert (TOKENS stages); nbuckets of them.
// Bytes left untouched after every workspace region (a canary a caller may
// check for writes past a region), and the most regions a layout has.
constexpr size_t kWsGuardBytes = 256;
constexpr int kMaxWsGuards = 24;
struct WsLayout {
    size_t chunk_counts;  // int32 [nchunks][nbuckets]
    size_t chunk_base;    // int32 [nchunks][nbuckets]
    size_t slot_rank;     // int32 [T*k]
    size_t ids;           // int32 [T*k]   (forward, when the caller passes none)
    size_t weights;       // fp32  [T*k]
    size_t logits;        // fp32  [T][E] router logits when E > 16 and T <= kRouteLogitsMaxTokens, else 0
                          // (chunk_counts is always at offset 0, so 0 means none)
    size_t counts;        // int32 [nbuckets] rows per bucket
    size_t counts_el;     // int32 [EL] rows per local expert (TOKENS stages)
    size_t offsets;       // int32 [nbuckets+1]
    size_t sorted_slot;   // int32 [Rcap]
    size_t slot_row;      // int32 [T*k]
    size_t x_perm;        // bf16  [Rcap][H] (0 bytes when no stage gathers)
    size_t act;           // bf16  [Rcap][I]
    size_t y_perm;        // fp32  [Rcap][H]
    size_t shared_act;    // bf16  [T][Is]
    size_t split_part;    // fp32  K-split partials (gemm_split_bytes; 0 bytes in exact order)
    size_t split_meta;    // int32 [kSplitMetaInts] K-split tail-tile records
    size_t split_part_sh; // the shared FFN's own K-split scratch when it may run beside
    size_t split_meta_sh; //   the routed GEMMs (0: it uses the one above)
    size_t total;
    int64_t nchunks;
    int64_t rcap;
    int nbuckets;
    // guard gaps of kWsGuardBytes after every region, never touched
    size_t guard[kMaxWsGuards];
    int nguards;
};
// Layout for moe_permute (o == NULL) or for moe_ffn_forward with options o
// (valid options: check them first).  shared_apart: the forward may run the
// shared FFN beside the routed GEMMs (its own streams), so their K splits
// need separate scratch; the no-allocation entry point runs one stream.
WsLayout ws_layout(const moe_dims *d, const moe_opts *o, bool shared_apart = true);
// The grouped gate/up GEMM can read its token rows straight from x through
// the dispatch order while every byte offset into x fits 32 bits.
bool gather_foldable(const moe_dims &d);
// Dispatch buckets moe_ffn_forward uses with options o (EL, or PN*EL for
// token-range stages); 0 when the options are not usable.
int forward_buckets(const moe_dims *d, const moe_opts *o);

// Permutation chunking: slots handled by one workgroup of the histogram pass.
constexpr int kPermChunk = 1024;

// K split of the grouped GEMM's last, partial round of tiles: at most
// kSplitMaxPieces pieces per tile, each at least kSplitMinStages K stages
// long (kSplitMinStagesAlone when the launch has fewer tiles than
// workgroups: decode-sized launches, whose pieces would otherwise leave
// most compute units idle while the weights stream), at most kSplitSlots
// pieces (partial-accumulator buffers) in all and kSplitMaxTail tiles cut.
// A launch of one partial round of more than half the grid spreads its K
// stages evenly over the grid instead (stream-K: a piece may end one tile
// and start the next).
constexpr int kSplitMaxPieces = 8;
constexpr int kSplitMinStages = 32;
constexpr int kSplitMinStagesAlone = 8;
constexpr int kSplitSlots = 512;
constexpr int kSplitMaxTail = 256;
constexpr int kSplitMetaInts = 4 + 4 * kSplitMaxTail;
// Bytes of the partial-accumulator buffer the grouped GEMM takes (all slots).
size_t gemm_split_bytes();

// Scratch of moe_ffn_forward_noalloc (a static device array per device).
constexpr size_t kNoAllocScratchBytes = size_t(256) << 20;

// ---- kernel launchers (stream-ordered, no host synchronisation) ----------
// logits: [T][E] fp32 scratch (may be NULL) for the many-expert, few-token
// path (E > 16, T <= kRouteLogitsMaxTokens).
constexpr int64_t kRouteLogitsMaxTokens = 4096;
// Up to this many waves (one per token and block of up to 16 experts) the
// router runs one chain per lane (few tokens: the chains' latency bounds
// the router); beyond, the lane-per-token kernels.
constexpr int64_t kRouteChainMaxWaves = 512;
hipError_t launch_route(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                        int32_t *ids, float *w, float *logits, hipStream_t s);
// Dispatch indices.  tokens_per_stage == 0: buckets are the local experts;
// else bucket = (t / tokens_per_stage) * EL + local expert and counts_el
// (may be NULL) receives the rows per local expert summed over stages.
hipError_t launch_permute(const moe_dims &d, const int32_t *ids, void *ws, const WsLayout &L,
                          int64_t tokens_per_stage, int32_t *counts, int32_t *offsets,
                          int32_t *counts_el, int32_t *sorted_slot, int32_t *slot_row,
                          hipStream_t s);
hipError_t launch_gather(const moe_dims &d, int e_first, int e_count, const int32_t *offsets,
                         const int32_t *sorted_slot, const bf16_t *x, bf16_t *x_perm,
                         int64_t max_rows, hipStream_t s);
// Combine of the local experts [e_first, e_first+e_count) for the tokens
// [t_begin, t_end).
hipError_t launch_combine(const moe_dims &d, int e_first, int e_count, int64_t t_begin,
                          int64_t t_end, const float *y_perm, const int32_t *ids,
                          const int32_t *slot_row, const float *w, float *y, int accumulate,
                          hipStream_t s);
// Grouped GEMMs over local experts [e_first, e_first+e_count) (rows from
// device offsets).  Gate/up takes its token rows either contiguous
// (row_map NULL: x_rows is x_perm) or straight from the token matrix
// (x_rows = x, row r is token row_map[r] / top_k, row_map = sorted_slot);
// the latter needs T*H*2 < 2^32 (byte offsets are 32-bit).
// parts / split_meta: gemm_split_bytes() and kSplitMetaInts int32 of
// scratch, or NULL: with them the tiles of the last, partial round of the
// persistent grid may be cut along K (then a fixup kernel follows the GEMM
// on the same stream); without them every tile is one pass over K.
// Launches that share the scratch must not overlap.
// bm: token rows of the tile, any valid_tile_rows value (every height
// gives the same bits in exact order); group_tile_rows picks it from a
// bound on the experts' row counts.  offsets NULL: a single expert
// (e_count 1) of rows_one contiguous rows, a count the host knows (the
// shared FFN over every token).
hipError_t launch_group_gateup(const moe_dims &d, int e_first, int e_count,
                               const int32_t *offsets, const bf16_t *x_rows,
                               const int32_t *row_map, const bf16_t *w_gate,
                               const bf16_t *w_up, bf16_t *act, int grid, float *parts,
                               int32_t *split_meta, int bm, hipStream_t s,
                               int64_t rows_one = 0);
hipError_t launch_group_down(const moe_dims &d, int e_first, int e_count,
                             const int32_t *offsets, const bf16_t *act,
                             const bf16_t *w_down, float *y_perm, int grid, float *parts,
                             int32_t *split_meta, int bm, hipStream_t s, int64_t rows_one = 0);
// Dense GEMMs over `rows` host-known contiguous rows, one tile per workgroup.
hipError_t launch_dense_gateup(int64_t rows, int H, int I, const bf16_t *x, const bf16_t *w_gate,
                               const bf16_t *w_up, bf16_t *act, int bm, hipStream_t s);
hipError_t launch_dense_down(int64_t rows, int H, int I, const bf16_t *act,
                             const bf16_t *w_down, float *y, int bm, hipStream_t s);

// ---- GEMM launch-cost model (host only) ----------------------------------
// Predicted microseconds of one persistent launch of `tiles` tiles of bm
// token rows over K (mode 0 gate/up, 1 down) on `grid` workgroups, with or
// without the K split of a partial last round.
double gemm_launch_us(int mode, int bm, int64_t tiles, int K, int grid, bool split);
// Tiles of one expert of `rows` rows: gate/up N = I (128 act columns per
// tile), down N = H (256 per tile).
int64_t gemm_tiles(int mode, int bm, int64_t rows, int N);
// Gate/up + down of one expert as two dense launches.
double ffn_expert_us(int bm, int64_t rows, int H, int I, int grid, bool split);
// The tile height the model prefers for a dense launch of `rows` rows.
int dense_tile_rows(int64_t rows, int H, int I, int grid, bool split);
// The tile height of a grouped launch none of whose experts has more than
// max_rows rows (the launch's tokens bound it: a token routes to an expert
// at most once): 320, or the smallest height that holds max_rows below it.
int group_tile_rows(int64_t max_rows);
// The tile height of a grouped launch over n_experts experts, none with more
// than max_rows rows: the launch-cost model prices each height up to
// group_tile_rows(max_rows) (gate/up over K = H, down over K = I) and the
// cheapest is taken when it is at least kGroupRowsMinGain below that
// height's price.  Shorter tiles pad less: for experts of a few rows each
// (decode batches, many experts) every tile is mostly padding, and the
// 128-row tile streams the weights faster.  rows: the experts' host row
// counts, or NULL when only the bound is known: then each expert's rows are
// taken as Binomial(tokens, p) (p = top_k / experts, uniform routing) and
// its tile counts as their expectation.
constexpr double kGroupRowsMinGain = 0.05;
int group_launch_rows(int64_t max_rows, const int32_t *rows, int n_experts, int64_t tokens,
                      double p, int H, int I, int grid, bool split);
// Skinny down GEMM for decode-sized grouped launches: one wave per tile of
// 64 output columns by an expert's rows (at most 64) over the whole K
// range, no K split (the same bits as every other tile height in exact
// order).  skinny_down_rows gives the tile's rows (16, 32 or 64) for a
// launch whose experts have at most max_rows rows, of which at most
// active_experts have any, with N output columns; 0 where the skinny tile
// does not apply: more rows, or fewer than two tiles per compute unit (the
// general tile's K split then keeps more loads in flight).
constexpr int64_t kSkinnyMaxRows = 64;
int skinny_down_rows(int64_t max_rows, int64_t active_experts, int N);
hipError_t launch_skinny_down(const moe_dims &d, int e_first, int e_count,
                              const int32_t *offsets, const bf16_t *act, const bf16_t *w_down,
                              float *y_perm, int bm, int64_t active_experts, hipStream_t s);
bool valid_tile_rows(int bm);

}  // namespace moe
