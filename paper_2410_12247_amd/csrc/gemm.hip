// Expert GEMMs of the SwiGLU FFN on gfx950 bf16 MFMA (fp32 accumulation).
//
// Two launches per expert group (the paper's Gate, Up and Down GEMMs, with
// the silu activation folded into the first):
//   gate/up : act[r][j] = bf16( silu(g) * u ),  g = Wg[j].x[r], u = Wu[j].x[r]
//   down    : y[r][h]   = Wd[h].act[r]                           (fp32 out)
// Both operands are contiguous along the reduced dimension.  The MFMA is
// fed the WEIGHT rows as its first (row) operand and the TOKEN rows as its
// second (column) operand, so each lane ends up holding four consecutive
// output features of one token row: a 16-byte fp32 store (down) or an
// 8-byte bf16 store (gate/up), and for gate/up the matching gate and up
// values sit in the same lane, so SiLU*mul needs no data movement.
//
// Workgroup tile (the one both schedulers use): 256 weight rows x 320 token
// rows, eight waves in two groups that alternate between MFMAs and memory
// work (the "ping-pong" tile below), built from v_mfma_f32_16x16x32_bf16.
// K advances 32 per stage through four LDS stages filled by LDS-DMA loads,
// so the loads of the next three stages are in flight while a stage is
// multiplied.  16-byte chunks of each LDS row are XOR-swizzled so MFMA
// operand reads hit distinct banks.  A four-wave tile (2 x 2 waves, one per
// SIMD, accumulators in AGPRs) is kept as the alternative selected with
// MOE_GEMM_PINGPONG=0; it is slower on the expert shapes measured.
//
// Two schedulers share that tile code and its arithmetic (so both give the
// same bits for the same rows):
//   dense : one launch per expert over host-known rows, one tile per
//           workgroup ("DenseGemm").
//   group : one persistent launch over a range of experts whose row counts
//           are read on the device; workgroups walk a tile list spanning
//           all experts ("GroupGemm").
// Both map workgroups to tiles XCD by XCD (the hardware deals workgroups
// round-robin over the 8 XCDs), so the tiles running on one XCD are
// neighbours in (m, n) and share activation and weight rows in its L2.
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "common.h"

namespace moe {
namespace {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

constexpr int NTHREADS = 256;
constexpr int NXCD = 8;
constexpr int GROUP_N = 8;  // n-tiles per super-column of the tile order

// XOR swizzle of the 16-byte chunk index inside an LDS row, chosen so that
// the 16 rows one MFMA operand read touches fall on distinct banks (LDS
// serves b128 reads eight lanes at a time): 128-byte rows (BK 64) use
// row & 7, 64-byte rows (BK 32) use (row >> 1) & 3.
template <int BK>
__device__ __forceinline__ int swz(int row) {
    return BK == 64 ? (row & 7) : ((row >> 1) & 3);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int MODE, int BN, int BM, int BK, int NS>
struct Cfg {
    static constexpr int WN = 2, WM = 2;
    static constexpr int WTN = BN / WN;  // weight rows per wave
    static constexpr int WTM = BM / WM;  // token rows per wave
    static constexpr int TN = WTN / 16;  // 16-row MFMA tiles along weights
    static constexpr int TM = WTM / 16;  // 16-row MFMA tiles along tokens
    static constexpr int CPR = BK / 8;   // 16-byte chunks per LDS row
    static constexpr int RPI = 64 / CPR; // rows one wave-wide LDS-DMA fills
    static constexpr int W_INSTR = BN / 4 / RPI;  // DMA instructions per wave per stage
    static constexpr int X_INSTR = BM / 4 / RPI;
    static constexpr int LPS = W_INSTR + X_INSTR;
    static constexpr int STAGE_W = BN * BK;  // bf16 elements per stage
    static constexpr int STAGE_X = BM * BK;
    static constexpr int STAGE = STAGE_W + STAGE_X;
    // output columns one tile covers: act columns (gate/up) or features (down)
    static constexpr int BNOUT = MODE == 0 ? BN / 2 : BN;
    static_assert((NS - 2) * LPS <= 63, "vmcnt range");
    static_assert(BN % (4 * RPI) == 0 && BM % (4 * RPI) == 0, "DMA tiling");
};

struct TileArgs {
    const bf16_t *w0;  // first weight row of the tile (gate rows, or down rows)
    const bf16_t *w1;  // first up row (gate/up only)
    int n_valid;       // weight rows valid from w0 (per half for gate/up)
    const bf16_t *x;   // first token row of the tile, or the token matrix
    const int32_t *rows;  // NULL: rows are contiguous from x; else tile row i
                          // is x row rows[i] / slot_div (the dispatch gather
                          // folded into the operand loads)
    int slot_div;
    int m_valid;       // token rows valid from x
    int K;             // row length of both operands (elements)
    int k0, nks;       // K stages [k0, k0 + nks) of BK elements this call covers
    void *out;         // output element (first token row, first column)
    int64_t ldo;       // output row stride in elements
    // K split (npieces > 1): this call is piece `piece` of the tile and
    // stores its fp32 accumulators in part[piece] instead of the output
    float *part;
    int piece, npieces;
};

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    __bf16 ha = static_cast<__bf16>(a);
    __bf16 hb = static_cast<__bf16>(b);
    uint16_t ua = __builtin_bit_cast(uint16_t, ha);
    uint16_t ub = __builtin_bit_cast(uint16_t, hb);
    return (uint32_t)ua | ((uint32_t)ub << 16);
}

// silu(g) * u = g * u / (1 + e^-g), with the hardware's exp2 and
// reciprocal (about 1 ulp each; the result is rounded to bf16 next):
// e^-g = 2^(-g log2 e).  An IEEE-rounded reciprocal costs a ten-instruction
// division sequence per value, and the gate/up epilogue evaluates 80 of
// them per lane with every wave of the workgroup in its epilogue at once.
// Large |g| behaves: e^-g -> inf gives 0 (silu -> 0), e^-g -> 0 gives g.
__device__ __forceinline__ float silu_mul(float g, float u) {
    const float e = __builtin_amdgcn_exp2f(g * -1.44269504088896341f);
    return g * __builtin_amdgcn_rcpf(1.0f + e) * u;
}

// One output tile.  Global -> LDS copies are wave-wide LDS-DMA loads
// (global_load_lds_dwordx4: lane l's 16 bytes land at base + 16*l, no
// registers involved); each wave fills its quarter of the weight and token
// rows of a stage.  NS stages are in flight: stage kt+NS-1 is requested
// while stage kt is multiplied, and a wave only waits (vmcnt) for the stage
// it needs next.
template <int MODE, int BN, int BM, int BK, int NS>
__device__ __forceinline__ void run_tile(const TileArgs &a, bf16_t *smem) {
    using C = Cfg<MODE, BN, BM, BK, NS>;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // wave index as a scalar: everything derived from it (LDS-DMA targets,
    // which weight half a wave copies) stays in SGPRs
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wn = wave % C::WN;
    const int wm = wave / C::WN;
    const int K = a.K;
    const int nk = K / BK;

    floatx4 acc[C::TN][C::TM];
#pragma unroll
    for (int t = 0; t < C::TN; ++t)
#pragma unroll
        for (int m = 0; m < C::TM; ++m) acc[t][m] = floatx4{0.f, 0.f, 0.f, 0.f};

    // ---- LDS-DMA assignment: this wave fills weight rows
    //      [wave*BN/4, (wave+1)*BN/4) and token rows [wave*BM/4, ...).
    const int drow = lane / C::CPR;                               // row within one DMA
    const int dchunk = ((lane % C::CPR) ^ swz<BK>(drow)) * 8;     // logical k offset
    const bf16_t *wsrc;
    int wrow0;
    if (MODE == 0) {
        // waves 0..1 copy gate rows, waves 2..3 copy up rows
        const bool up = wave >= 2;
        wsrc = up ? a.w1 : a.w0;
        wrow0 = (wave & 1) * (BN / 4);
    } else {
        wsrc = a.w0;
        wrow0 = wave * (BN / 4);
    }
    // per-lane byte offsets from the (scalar) tile base; rows past the valid
    // range read a valid row, whose results are never stored
    uint32_t woff[C::W_INSTR];
#pragma unroll
    for (int i = 0; i < C::W_INSTR; ++i) {
        const int r = min(wrow0 + i * C::RPI + drow, a.n_valid - 1);
        woff[i] = (uint32_t)(r * K + dchunk) * 2u;
    }
    uint32_t xoff[C::X_INSTR];
#pragma unroll
    for (int i = 0; i < C::X_INSTR; ++i) {
        const int r = min(wave * (BM / 4) + i * C::RPI + drow, a.m_valid - 1);
        const int64_t src = a.rows ? (int64_t)(a.rows[r] / a.slot_div) : r;
        xoff[i] = (uint32_t)((src * K + dchunk) * 2);
    }
    const int w_lds = wave * (BN / 4) * BK;  // element offset of this wave's rows
    const int x_lds = C::STAGE_W + wave * (BM / 4) * BK;

    // scalar base + per-lane 32-bit offset: the SADDR form of the load
    auto issue = [&](int stage, int k0) {
        bf16_t *sb = smem + stage * C::STAGE;
        const char *wk = reinterpret_cast<const char *>(wsrc + k0);
        const char *xk = reinterpret_cast<const char *>(a.x + k0);
#pragma unroll
        for (int i = 0; i < C::W_INSTR; ++i)
            __builtin_amdgcn_global_load_lds((gbl_void_t *)(wk + woff[i]),
                                             (lds_void_t *)(sb + w_lds + i * C::RPI * BK), 16,
                                             0, 0);
#pragma unroll
        for (int i = 0; i < C::X_INSTR; ++i)
            __builtin_amdgcn_global_load_lds((gbl_void_t *)(xk + xoff[i]),
                                             (lds_void_t *)(sb + x_lds + i * C::RPI * BK), 16,
                                             0, 0);
    };

    // ---- fragment rows (LDS row of lane 0 of each 16-row MFMA tile)
    int arow[C::TN];
#pragma unroll
    for (int t = 0; t < C::TN; ++t) {
        if (MODE == 0) {
            arow[t] = t < C::TN / 2 ? wn * (C::WTN / 2) + t * 16
                                    : BN / 2 + wn * (C::WTN / 2) + (t - C::TN / 2) * 16;
        } else {
            arow[t] = wn * C::WTN + t * 16;
        }
    }
    const int lrow = lane & 15;
    const int lk = lane >> 4;  // which 8-wide k group of the 32-wide MFMA step
    const int lsw = swz<BK>(lrow);

    // Operand fragments are double-buffered in registers: while the MFMAs
    // of stage kt run, the fragments of stage kt+1 are read from LDS.
    struct Frags {
        bf16x8 a[C::TN];
        bf16x8 b[C::TM];
    };
    static_assert(BK == 32, "one 32-wide MFMA step per stage");
    static_assert(NS == 4, "the K loop below is unrolled for four stages");
    Frags f0, f1;

    auto load_frags = [&](int stage, Frags &f) {
        const bf16_t *sw = smem + stage * C::STAGE;
        const bf16_t *sx = sw + C::STAGE_W;
        const int chunk = (lk ^ lsw) * 8;
#pragma unroll
        for (int t = 0; t < C::TN; ++t)
            f.a[t] = *reinterpret_cast<const bf16x8 *>(sw + (arow[t] + lrow) * BK + chunk);
#pragma unroll
        for (int m = 0; m < C::TM; ++m)
            f.b[m] = *reinterpret_cast<const bf16x8 *>(
                sx + (wm * C::WTM + m * 16 + lrow) * BK + chunk);
    };
    auto mfmas = [&](const Frags &f) {
#pragma unroll
        for (int m = 0; m < C::TM; ++m)
#pragma unroll
            for (int t = 0; t < C::TN; ++t)
                acc[t][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[t], f.b[m], acc[t][m],
                                                                    0, 0, 0);
    };
    // one LDS read issued between every (TN*TM)/(TN+TM) MFMAs
    auto interleave = [&]() {
        constexpr int NREAD = C::TN + C::TM;
        constexpr int PER = (C::TN * C::TM) / NREAD;
#pragma unroll
        for (int i = 0; i < NREAD; ++i) {
            if (i < C::LPS) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);                  // DS read
            __builtin_amdgcn_sched_group_barrier(0x008, PER, 0);                // MFMA
        }
    };
    // stage kt lives in LDS buffer u = kt % NS and in register set cur
    auto step = [&](int kt, int u, Frags &cur, Frags &nxt) {
        const bool ahead = kt + NS - 1 < nk;
        // Stage kt+NS-1 is requested unconditionally (past the end it re-reads
        // the last stage into a buffer that is never read again), so the
        // loads, LDS reads and MFMAs form one block the scheduler interleaves.
        issue((u + NS - 1) % NS, (ahead ? kt + NS - 1 : nk - 1) * BK);
        // the prefetch of stage kt+1 is unconditional: past the last stage it
        // reads a stale (in-bounds) LDS buffer whose values are never used,
        // which keeps a single MFMA block (accumulators stay in AGPRs)
        load_frags((u + 1) % NS, nxt);
        mfmas(cur);
        interleave();
        if (kt + 2 < nk) {
            // stage kt+2 must be in LDS (every wave's share) before the next
            // step reads it
            if (ahead) wait_vmcnt<(NS - 3) * C::LPS>(); else wait_vmcnt<0>();
            __builtin_amdgcn_s_barrier();
        }
    };

    // prologue: stages 0..NS-2 requested; stage 0 in registers, stage 1 in LDS
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
        if (s < nk) issue(s, s * BK);
    if (nk >= NS - 1) wait_vmcnt<(NS - 2) * C::LPS>(); else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    load_frags(0, f0);
    if (nk >= NS - 1) wait_vmcnt<(NS - 3) * C::LPS>(); else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();

    for (int kt0 = 0; kt0 < nk; kt0 += NS) {
        step(kt0, 0, f0, f1);
        if (kt0 + 1 < nk) step(kt0 + 1, 1, f1, f0);
        if (kt0 + 2 < nk) step(kt0 + 2, 2, f0, f1);
        if (kt0 + 3 < nk) step(kt0 + 3, 3, f1, f0);
    }
    __builtin_amdgcn_s_barrier();  // LDS free for the next tile of this workgroup

    // ---- epilogue: lane holds output columns col..col+3 of token row `row`
    const int lcol4 = (lane >> 4) * 4;
    if (MODE == 0) {
        bf16_t *out = reinterpret_cast<bf16_t *>(a.out);
#pragma unroll
        for (int t = 0; t < C::TN / 2; ++t) {
            const int col = wn * (C::WTN / 2) + t * 16 + lcol4;
#pragma unroll
            for (int m = 0; m < C::TM; ++m) {
                const int row = wm * C::WTM + m * 16 + lrow;
                if (row < a.m_valid && col < a.n_valid) {
                    const floatx4 g = acc[t][m];
                    const floatx4 u = acc[t + C::TN / 2][m];
                    uint2 v;
                    v.x = pack_bf16x2(silu_mul(g[0], u[0]), silu_mul(g[1], u[1]));
                    v.y = pack_bf16x2(silu_mul(g[2], u[2]), silu_mul(g[3], u[3]));
                    *reinterpret_cast<uint2 *>(out + row * a.ldo + col) = v;
                }
            }
        }
    } else {
        float *out = reinterpret_cast<float *>(a.out);
#pragma unroll
        for (int t = 0; t < C::TN; ++t) {
            const int col = wn * C::WTN + t * 16 + lcol4;
#pragma unroll
            for (int m = 0; m < C::TM; ++m) {
                const int row = wm * C::WTM + m * 16 + lrow;
                if (row < a.m_valid && col < a.n_valid)
                    *reinterpret_cast<floatx4 *>(out + row * a.ldo + col) = acc[t][m];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Eight-wave ping-pong variant.  256 (weights) x BM (tokens) output tile,
// eight waves in two groups of four, one wave of each group on every SIMD.
// Each wave owns a 128 x BM/4 accumulator block.  The groups alternate
// between a compute phase (MFMAs on fragments already in registers) and a
// memory phase (its share of the LDS-DMA for stage k+NS-1 and the fragment
// reads of its next stage), separated by workgroup barriers, so every SIMD
// always has one wave issuing MFMAs while the other feeds LDS.  Stage s
// lives in LDS buffer s % NS (NS = 4 stages of 32 K, or 3 of 64 K).
//   group A (waves 0-3, token rows 0..BM/2-1):  compute(k) | mem: frags(k+1), DMA(k+NS-1)
//   group B (waves 4-7, token rows BM/2..BM-1): mem: frags(k), DMA(k+NS-1) | compute(k)
// LDS traffic per MFMA falls as the wave tile grows: BM = 320 (wave tile
// 128 x 80, 40 MFMAs per 13 fragment reads, 160 accumulator registers, four
// 36 KiB stages) is the largest that fits 256 registers and 160 KiB of LDS.
// ---------------------------------------------------------------------------
constexpr int PP_THREADS = 512;
// K per LDS stage of the ping-pong tile of bm token rows: 64 for the
// 128-row tile (decode-sized launches, bound by the weight stream, read 128
// contiguous bytes of each weight row per stage instead of 64: about 10%
// faster on 64-token decode), 32 for the taller, MFMA-bound tiles
__host__ __device__ constexpr int pp_stage_k(int bm) { return bm == 128 ? 64 : 32; }
// buffer resource word 3 for raw (untyped, unswizzled) access on gfx9 parts
constexpr int kBufferFlags = 0x00020000;

template <int MODE, int BM_>
struct PPCfg {
    static constexpr int BN = 256, BM = BM_;
    static constexpr int BK = pp_stage_k(BM_);
    static constexpr int NS = BK == 64 ? 3 : 4;  // ring within 144 KB of LDS
    static constexpr int KH = BK / 32;  // MFMA K-steps per stage
    static constexpr int WTN = 128, WTM = BM / 4;  // wave tile (weights x tokens)
    static constexpr int TN = WTN / 16, TM = WTM / 16;
    static_assert(WTM % 16 == 0, "token rows per wave: whole 16-row fragments");
    static constexpr int CPR = BK / 8;          // 16-byte chunks per LDS row
    static constexpr int RPI = 64 / CPR;        // rows one LDS-DMA instruction fills
    static constexpr int W_INSTR = BN / 8 / RPI;
    // token rows: BM / RPI instructions, group A's waves take X_INSTR_A
    // each, group B's the rest
    static constexpr int X_TOTAL = BM / RPI;
    static constexpr int X_INSTR_A = (X_TOTAL + 7) / 8;
    static constexpr int X_INSTR_B = (X_TOTAL - 4 * X_INSTR_A) / 4;
    static_assert(4 * X_INSTR_A + 4 * X_INSTR_B == X_TOTAL, "token rows split over waves");
    static constexpr int LPS_A = W_INSTR + X_INSTR_A;  // DMA instructions per wave per stage
    static constexpr int LPS_B = W_INSTR + X_INSTR_B;
    static constexpr int STAGE_W = BN * BK, STAGE_X = BM * BK, STAGE = STAGE_W + STAGE_X;
    static constexpr int LDS_ELEMS = NS * STAGE;
    static_assert(LDS_ELEMS * 2 <= 144 * 1024, "ring within 144 KB of LDS");
    static_assert(NS >= 3 && (NS - 2) * (LPS_A > LPS_B ? LPS_A : LPS_B) <= 63, "vmcnt range");
    static constexpr int BNOUT = MODE == 0 ? BN / 2 : BN;
    static constexpr int PART_ELEMS = BN * BM;  // fp32 accumulators of one tile
    static constexpr int PART_BYTES = PART_ELEMS * 4;
    static constexpr int WAVE_BYTES = TN * TM * 1024;  // one wave's block of them
};

// Epilogue of a ping-pong tile (or of the sum of its K pieces), one 16x16
// output fragment at a time; the lane holds output columns col..col+3 of
// token row `row`.  gate/up: fragment (p, m) of wave (wn, wm) from the
// matching gate and up accumulators, stored as bf16(silu(g) * u).
template <class C>
__device__ __forceinline__ void store_gateup(const floatx4 &g, const floatx4 &u, int p, int m,
                                             int wn, int wm, int lane, bf16_t *out, int64_t ldo,
                                             int m_valid, int n_valid) {
    const int row = wm * C::WTM + m * 16 + (lane & 15);
    const int col = wn * (C::WTN / 2) + p * 16 + (lane >> 4) * 4;
    if (row < m_valid && col < n_valid) {
        uint2 v;
        v.x = pack_bf16x2(silu_mul(g[0], u[0]), silu_mul(g[1], u[1]));
        v.y = pack_bf16x2(silu_mul(g[2], u[2]), silu_mul(g[3], u[3]));
        *reinterpret_cast<uint2 *>(out + row * ldo + col) = v;
    }
}
// down: fragment (t, m) of wave (wn, wm), the fp32 values.
template <class C>
__device__ __forceinline__ void store_down(const floatx4 &v, int t, int m, int wn, int wm,
                                           int lane, float *out, int64_t ldo, int m_valid,
                                           int n_valid) {
    const int row = wm * C::WTM + m * 16 + (lane & 15);
    const int col = wn * C::WTN + t * 16 + (lane >> 4) * 4;
    if (row < m_valid && col < n_valid) *reinterpret_cast<floatx4 *>(out + row * ldo + col) = v;
}

template <int MODE, class C>
__device__ __forceinline__ void pp_epilogue(const floatx4 (&acc)[C::TN][C::TM], int wn, int wm,
                                            int lane, void *outp, int64_t ldo, int m_valid,
                                            int n_valid) {
    if (MODE == 0) {
#pragma unroll
        for (int p = 0; p < C::TN / 2; ++p)
#pragma unroll
            for (int m = 0; m < C::TM; ++m)
                store_gateup<C>(acc[p][m], acc[p + C::TN / 2][m], p, m, wn, wm, lane,
                                reinterpret_cast<bf16_t *>(outp), ldo, m_valid, n_valid);
    } else {
#pragma unroll
        for (int t = 0; t < C::TN; ++t)
#pragma unroll
            for (int m = 0; m < C::TM; ++m)
                store_down<C>(acc[t][m], t, m, wn, wm, lane, reinterpret_cast<float *>(outp), ldo,
                              m_valid, n_valid);
    }
}

template <int MODE, int BM_>
__device__ __forceinline__ void run_tile_pp(const TileArgs &a, bf16_t *smem) {
    using C = PPCfg<MODE, BM_>;
    constexpr int BK = C::BK, NS = C::NS;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wave >> 2;  // 0 = A, 1 = B
    const int wn = wave & 1;    // weight half
    const int wm = wave >> 1;   // 64-row token block
    const int K = a.K;
    const int nk = a.nks;
    // a wave whose token rows or weight rows all lie past the valid edge of
    // a partial tile skips its MFMAs (its outputs are never stored); it still
    // takes its share of the loads and barriers
    const bool active = wm * C::WTM < a.m_valid &&
                        (MODE == 0 ? wn * (C::WTN / 2) : wn * C::WTN) < a.n_valid;

    floatx4 acc[C::TN][C::TM];
#pragma unroll
    for (int t = 0; t < C::TN; ++t)
#pragma unroll
        for (int m = 0; m < C::TM; ++m) acc[t][m] = floatx4{0.f, 0.f, 0.f, 0.f};

    // ---- LDS-DMA share of this wave: BN/8 weight rows and a slice of the
    // token rows (BM/16 instructions of 16 rows split over the waves,
    // group A's waves taking the larger slices when they do not divide evenly)
    const int drow = lane / C::CPR;
    const int dchunk = ((lane % C::CPR) ^ swz<BK>(drow)) * 8;
    const bf16_t *wsrc;
    int wrow0;
    if (MODE == 0) {  // waves 0..3 copy gate rows, 4..7 up rows
        wsrc = wave >= 4 ? a.w1 : a.w0;
        wrow0 = (wave & 3) * (C::BN / 8);
    } else {
        wsrc = a.w0;
        wrow0 = wave * (C::BN / 8);
    }
    uint32_t woff[C::W_INSTR], xoff[C::X_INSTR_A];
#pragma unroll
    for (int i = 0; i < C::W_INSTR; ++i) {
        const int r = min(wrow0 + i * C::RPI + drow, a.n_valid - 1);
        woff[i] = (uint32_t)(r * K + dchunk) * 2u;
    }
    // first token row of this wave's LDS-DMA share
    const int x_row0 = grp == 0 ? wave * C::X_INSTR_A * C::RPI
                                : 4 * C::X_INSTR_A * C::RPI + (wave - 4) * C::X_INSTR_B * C::RPI;
#pragma unroll
    for (int i = 0; i < C::X_INSTR_A; ++i) {
        const int r = min(x_row0 + i * C::RPI + drow, a.m_valid - 1);
        const int64_t src = a.rows ? (int64_t)(a.rows[r] / a.slot_div) : r;
        xoff[i] = (uint32_t)((src * K + dchunk) * 2);
    }
    const int w_lds = wave * (C::BN / 8) * BK;
    const int x_lds = C::STAGE_W + x_row0 * BK;
    // this wave's share of stage kstage (clamped); nx: its token-row
    // instruction count (the group's)
    // buffer resources over the weight rows and the token rows: a 32-bit
    // per-lane row offset plus the stage's k offset as the scalar offset
    const __amdgpu_buffer_rsrc_t wres =
        __builtin_amdgcn_make_buffer_rsrc((void *)wsrc, 0, -1, kBufferFlags);
    const __amdgpu_buffer_rsrc_t xres =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, 0, -1, kBufferFlags);
    auto issue = [&](int kstage, auto nx) {
        const int ks = min(kstage, nk - 1);
        bf16_t *sb = smem + (kstage % NS) * C::STAGE;
        const int kb = (a.k0 + ks) * BK * 2;
#pragma unroll
        for (int i = 0; i < C::W_INSTR; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                wres, (lds_void_t *)(sb + w_lds + i * C::RPI * BK), 16, woff[i], kb, 0, 0);
#pragma unroll
        for (int i = 0; i < decltype(nx)::value; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                xres, (lds_void_t *)(sb + x_lds + i * C::RPI * BK), 16, xoff[i], kb, 0, 0);
    };

    // ---- fragments of this wave
    int arow[C::TN];
#pragma unroll
    for (int t = 0; t < C::TN; ++t) {
        if (MODE == 0)
            arow[t] = t < C::TN / 2 ? wn * (C::WTN / 2) + t * 16
                                    : C::BN / 2 + wn * (C::WTN / 2) + (t - C::TN / 2) * 16;
        else
            arow[t] = wn * C::WTN + t * 16;
    }
    const int lrow = lane & 15;
    // the chunk holding K 32 h + 8 (lane / 16) .. + 7 of a row, K-step h
    int chunk[C::KH];
#pragma unroll
    for (int h = 0; h < C::KH; ++h) chunk[h] = ((h * 4 + (lane >> 4)) ^ swz<BK>(lrow)) * 8;
    bf16x8 fa[C::KH][C::TN], fb[C::KH][C::TM];
    auto load_frags = [&](int kstage) {  // stale but in-bounds past the end
        const bf16_t *sw = smem + (kstage % NS) * C::STAGE;
        const bf16_t *sx = sw + C::STAGE_W;
#pragma unroll
        for (int h = 0; h < C::KH; ++h) {
#pragma unroll
            for (int t = 0; t < C::TN; ++t)
                fa[h][t] =
                    *reinterpret_cast<const bf16x8 *>(sw + (arow[t] + lrow) * BK + chunk[h]);
#pragma unroll
            for (int m = 0; m < C::TM; ++m)
                fb[h][m] = *reinterpret_cast<const bf16x8 *>(
                    sx + (wm * C::WTM + m * 16 + lrow) * BK + chunk[h]);
        }
    };
    auto mfmas = [&]() {  // K-steps in ascending order
#pragma unroll
        for (int h = 0; h < C::KH; ++h)
#pragma unroll
            for (int m = 0; m < C::TM; ++m)
#pragma unroll
                for (int t = 0; t < C::TN; ++t)
                    acc[t][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[h][t], fb[h][m],
                                                                        acc[t][m], 0, 0, 0);
    };

    // prologue: stages 0 .. NS-2 requested by every wave, all landed
    using nxa = std::integral_constant<int, C::X_INSTR_A>;
    using nxb = std::integral_constant<int, C::X_INSTR_B>;
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) {
        if (grp == 0) issue(s, nxa{}); else issue(s, nxb{});
    }
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();

    // the two groups' loops, with or without the MFMAs; each is straight
    // code (no branch around the MFMA block inside the loop)
    auto loop_a = [&](auto with_mfma) {
        load_frags(0);
        for (int k = 0; k < nk; ++k) {
            // compute phase: stage k
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __builtin_amdgcn_s_setprio(1);
            if constexpr (decltype(with_mfma)::value) mfmas();
            __builtin_amdgcn_s_setprio(0);
            // stage k+1 landed before the barrier; this wave's requests for
            // stages k+2 .. k+NS-2 may stay in flight
            wait_vmcnt<(NS - 3) * C::LPS_A>();
            __builtin_amdgcn_s_barrier();
            // memory phase: fragments of stage k+1, this wave's share of stage k+NS-1
            load_frags(k + 1);
            issue(k + NS - 1, nxa{});
            __builtin_amdgcn_s_barrier();
        }
    };
    auto loop_b = [&](auto with_mfma) {
        for (int k = 0; k < nk; ++k) {
            // memory phase: fragments of stage k, this wave's share of stage k+NS-1
            load_frags(k);
            issue(k + NS - 1, nxb{});
            // stage k+1 landed; this wave's requests for stages k+2 ..
            // k+NS-1 (the last just issued) may stay in flight
            wait_vmcnt<(NS - 2) * C::LPS_B>();
            __builtin_amdgcn_s_barrier();
            // compute phase: stage k
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __builtin_amdgcn_s_setprio(1);
            if constexpr (decltype(with_mfma)::value) mfmas();
            __builtin_amdgcn_s_setprio(0);
            __builtin_amdgcn_s_barrier();
        }
    };
    using on = std::integral_constant<bool, true>;
    using off = std::integral_constant<bool, false>;
    if (grp == 0) {
        if (active) loop_a(on{}); else loop_a(off{});
    } else {
        if (active) loop_b(on{}); else loop_b(off{});
    }
    wait_vmcnt<0>();  // clamped tail requests drained before LDS is reused
    __builtin_amdgcn_s_barrier();

    // ---- K split: the piece stores its accumulators (each wave its own
    // block, one 1 KiB store per fragment, through a buffer resource so the
    // fragment offsets are scalars); split_fixup_kernel adds the pieces and
    // runs the epilogue
    if (a.npieces > 1) {
        const __amdgpu_buffer_rsrc_t pres =
            __builtin_amdgcn_make_buffer_rsrc(a.part, 0, -1, kBufferFlags);
        const int loff = lane * 16;
        // fragment rows wholly past the valid edge are never stored, so
        // their partial sums are neither written nor read back (decode-sized
        // tiles hold one or two valid rows of 320)
#pragma unroll
        for (int m = 0; m < C::TM; ++m) {
            if (wm * C::WTM + m * 16 >= a.m_valid) break;
#pragma unroll
            for (int t = 0; t < C::TN; ++t)
                __builtin_amdgcn_raw_buffer_store_b128(
                    __builtin_bit_cast(u32x4, acc[t][m]), pres, loff,
                    a.piece * C::PART_BYTES + wave * C::WAVE_BYTES + (t * C::TM + m) * 1024, 0);
        }
        return;
    }

    pp_epilogue<MODE, C>(acc, wn, wm, lane, a.out, a.ldo, a.m_valid, a.n_valid);
}

// Tile order inside one expert: super-columns of GROUP_N n-tiles, walked
// row by row, so consecutive tiles share token rows and weight rows.
__device__ __forceinline__ void decode_tile(int tau, int MT, int NT, int &mt, int &nt) {
    const int per_sc = GROUP_N * MT;
    const int sc = tau / per_sc;
    const int r = tau - sc * per_sc;
    const int width = min(GROUP_N, NT - sc * GROUP_N);
    mt = r / width;
    nt = sc * GROUP_N + (r - mt * width);
}

// Tile policies shared by the two schedulers.
template <int MODE, int BN_, int BM_, int BK, int NS>
struct FourWave {
    using C = Cfg<MODE, BN_, BM_, BK, NS>;
    static constexpr int THREADS = NTHREADS;
    static constexpr int BM = BM_;
    static constexpr int BNOUT = C::BNOUT;
    static constexpr int LDS_ELEMS = NS * C::STAGE;
    static constexpr int KSTEP = BK;
    static constexpr bool CAN_SPLIT = false;  // covers the whole K range only
    static constexpr int PART_ELEMS = 0;
    static __device__ __forceinline__ void run(const TileArgs &a, bf16_t *smem) {
        run_tile<MODE, BN_, BM_, BK, NS>(a, smem);
    }
};
template <int MODE, int BM_>
struct PingPong {
    using C = PPCfg<MODE, BM_>;  // also read by split_fixup_kernel
    static constexpr int THREADS = PP_THREADS;
    static constexpr int BM = C::BM;
    static constexpr int BNOUT = C::BNOUT;
    static constexpr int LDS_ELEMS = C::LDS_ELEMS;
    static constexpr int KSTEP = C::BK;
    static constexpr bool CAN_SPLIT = true;
    static constexpr int PART_ELEMS = C::PART_ELEMS;
    static __device__ __forceinline__ void run(const TileArgs &a, bf16_t *smem) {
        run_tile_pp<MODE, BM_>(a, smem);
    }
};

template <int MODE, class TP>
__global__ __launch_bounds__(TP::THREADS) void dense_kernel(const bf16_t *__restrict__ x,
                                                            int64_t rows, const bf16_t *w0,
                                                            const bf16_t *w1, int N, int K,
                                                            void *out, int64_t ldo, int MT,
                                                            int NT) {
    constexpr int BM = TP::BM;
    __shared__ __attribute__((aligned(16))) bf16_t smem[TP::LDS_ELEMS];
    const int per = gridDim.x / NXCD;
    const int tau = (blockIdx.x % NXCD) * per + blockIdx.x / NXCD;
    if (tau >= MT * NT) return;
    int mt, nt;
    decode_tile(tau, MT, NT, mt, nt);
    TileArgs a;
    const int64_t n0 = (int64_t)nt * TP::BNOUT;
    const int64_t m0 = (int64_t)mt * BM;
    a.w0 = w0 + n0 * K;
    a.w1 = MODE == 0 ? w1 + n0 * K : nullptr;
    a.n_valid = (int)(N - n0);
    a.x = x + m0 * K;
    a.rows = nullptr;
    a.slot_div = 1;
    a.m_valid = (int)min<int64_t>(BM, rows - m0);
    a.K = K;
    a.k0 = 0;
    a.nks = K / TP::KSTEP;
    a.ldo = ldo;
    a.part = nullptr;
    a.piece = 0;
    a.npieces = 1;
    if (MODE == 0)
        a.out = reinterpret_cast<bf16_t *>(out) + m0 * ldo + n0;
    else
        a.out = reinterpret_cast<float *>(out) + m0 * ldo + n0;
    TP::run(a, smem);
}

template <int MODE, class TP>
__global__ __launch_bounds__(TP::THREADS) void group_kernel(
    const int32_t *__restrict__ offsets, int e_first, int e_count, const bf16_t *__restrict__ x,
    const int32_t *__restrict__ row_map, int slot_div, const bf16_t *w0s, const bf16_t *w1s,
    int64_t wstride, int N, int K, void *out, int64_t ldo, float *__restrict__ parts,
    int32_t *__restrict__ split_meta, int rows_one) {
    constexpr int BM = TP::BM;
    // one LDS object (stage buffers, then the per-expert offsets and tile
    // prefix sums): the compiler then does not make fragment reads wait for
    // the LDS-DMA in flight
    __shared__ __attribute__((aligned(16))) bf16_t smem[TP::LDS_ELEMS + 4 * (kMaxExperts + 1)];
    int *s_off = reinterpret_cast<int *>(smem + TP::LDS_ELEMS);
    int *s_pre = s_off + (kMaxExperts + 1);
    const int tid = threadIdx.x;
    const int NT = (N + TP::BNOUT - 1) / TP::BNOUT;

    // offsets NULL: one expert of rows_one rows (known on the host)
    for (int i = tid; i <= e_count; i += TP::THREADS)
        s_off[i] = offsets ? offsets[e_first + i] : (i == 0 ? 0 : rows_one);
    __syncthreads();
    // tiles per expert, then an inclusive scan (Hillis-Steele over <= 256)
    int mine = 0;
    if (tid < e_count) mine = ((s_off[tid + 1] - s_off[tid] + BM - 1) / BM) * NT;
    if (tid < kMaxExperts) s_pre[tid + 1] = mine;
    if (tid == 0) s_pre[0] = 0;
    __syncthreads();
    for (int d = 1; d < kMaxExperts; d <<= 1) {
        int v = 0;
        if (tid < kMaxExperts && tid >= d) v = s_pre[tid + 1 - d];
        __syncthreads();
        if (tid < kMaxExperts) s_pre[tid + 1] += v;
        __syncthreads();
    }
    const int total = s_pre[e_count];

    const int G = gridDim.x;  // multiple of NXCD
    const int slot = (blockIdx.x % NXCD) * (G / NXCD) + blockIdx.x / NXCD;
    const int nk = K / TP::KSTEP;
    // Tiles [0, full) fill whole rounds of the grid.  The rem < G tiles left
    // would occupy rem workgroups for one more tile time while the others
    // idle.  With a split buffer the tail is cut along K:
    //  - rem <= G/2: each tail tile j = tau - full into S equal pieces
    //    (slots [S*j, S*j + S));
    //  - a launch that is one partial round of more than G/2 tiles (full ==
    //    0): its W = rem * nk K stages, the tail tiles laid end to end, are
    //    spread evenly over P <= G units (stream-K): unit u takes stages
    //    [u*W/P, (u+1)*W/P), so it ends one tile and starts the next, and its
    //    segment of tile j goes to slot u + j (unique: a unit that reaches
    //    into tile j + 1 is the last of tile j).  Only for tiles of 192 or
    //    more token rows (their MFMA work, done for every row of the tile,
    //    bounds them; a round of 128-row tiles is bound by the weight
    //    stream, which fewer workgroups already saturate), at most half
    //    full on average (each piece writes and the fixup re-reads the
    //    partial sums of the valid rows: for fuller tiles that traffic
    //    outweighs the shorter round), and when the round gets at least a
    //    quarter shorter.
    // The pieces store fp32 partial sums; split_fixup_kernel, launched next,
    // adds each tile's pieces in K order and writes the outputs.
    // split_meta: [0] tail tiles cut (0: none), [1] S (0: stream-K), [2] P,
    // [3] nk, then per tail tile its first output row, first output column
    // and valid rows and columns.
    const int full = total - total % G;
    const int rem = total - full;
    const int64_t W = (int64_t)rem * nk;
    int S = 1, P = 0;
    if (TP::CAN_SPLIT && parts != nullptr && rem > 0 && rem <= kSplitMaxTail) {
        if (full == 0 && 2 * rem > G && BM >= 192) {
            // mean valid rows per tile: all rows over the m-tiles
            const int64_t rows_all = s_off[e_count] - s_off[0];
            if (2 * rows_all * NT <= (int64_t)BM * total) {
                P = (int)min<int64_t>(min(G, kSplitSlots - rem), W / kSplitMinStagesAlone);
                if (4 * rem > 3 * P) P = 0;
            }
        } else {
            S = min(min(kSplitMaxPieces, G / rem),
                    min(nk / (full == 0 ? kSplitMinStagesAlone : kSplitMinStages),
                        kSplitSlots / rem));
        }
    }
    if (S < 2) S = 1;
    if (split_meta != nullptr && slot == 0 && tid == 0) {
        split_meta[0] = S > 1 || P > 0 ? rem : 0;
        split_meta[1] = P > 0 ? 0 : S;
        split_meta[2] = P;
        split_meta[3] = nk;
    }

    // tile tau over K stages [k0, k0 + nks); part: the slot of its partial
    // sums (NULL: the whole K range, outputs written); j >= 0: the tail tile
    // whose record this call writes (the call that starts at stage 0)
    auto run_tau = [&](int tau, int k0, int nks, float *part, int j) {
        // expert: last e with s_pre[e] <= tau
        int lo = 0, hi = e_count - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_pre[mid] <= tau) lo = mid; else hi = mid - 1;
        }
        const int e = lo;
        const int cnt = s_off[e + 1] - s_off[e];
        const int MT = (cnt + BM - 1) / BM;
        int mt, nt;
        decode_tile(tau - s_pre[e], MT, NT, mt, nt);
        const int64_t n0 = (int64_t)nt * TP::BNOUT;
        const int64_t r0 = (int64_t)s_off[e] + (int64_t)mt * BM;
        TileArgs a;
        const int64_t woffe = (int64_t)(e_first + e) * wstride;
        a.w0 = w0s + woffe + n0 * K;
        a.w1 = MODE == 0 ? w1s + woffe + n0 * K : nullptr;
        a.n_valid = (int)(N - n0);
        a.x = row_map ? x : x + r0 * K;
        a.rows = row_map ? row_map + r0 : nullptr;
        a.slot_div = slot_div;
        a.m_valid = min(BM, cnt - mt * BM);
        a.K = K;
        a.k0 = k0;
        a.nks = nks;
        a.ldo = ldo;
        if (MODE == 0)
            a.out = reinterpret_cast<bf16_t *>(out) + r0 * ldo + n0;
        else
            a.out = reinterpret_cast<float *>(out) + r0 * ldo + n0;
        a.part = part;
        a.piece = 0;
        a.npieces = part != nullptr ? 2 : 1;
        if (j >= 0 && tid == 0) {
            int32_t *md = split_meta + 4 + 4 * j;
            md[0] = (int32_t)r0;
            md[1] = (int32_t)n0;
            md[2] = a.m_valid;
            md[3] = a.n_valid;
        }
        TP::run(a, smem);
    };

    if (P > 0) {
        // stream-K tail (full == 0): at most one unit per workgroup
        if (slot < P) {
            const int64_t g0 = (int64_t)slot * W / P, g1 = (int64_t)(slot + 1) * W / P;
            for (int j = (int)(g0 / nk); (int64_t)j * nk < g1; ++j) {
                const int64_t a0 = max<int64_t>(g0, (int64_t)j * nk);
                const int64_t a1 = min<int64_t>(g1, (int64_t)(j + 1) * nk);
                run_tau(j, (int)(a0 - (int64_t)j * nk), (int)(a1 - a0),
                        parts + (size_t)(slot + j) * TP::PART_ELEMS, a0 == (int64_t)j * nk ? j : -1);
            }
        }
        return;
    }
    const int end = S > 1 ? full : total;
    const int units = S > 1 ? full + rem * S : total;
    for (int u = slot; u < units; u += G) {
        if (u < end) {
            run_tau(u, 0, nk, nullptr, -1);
        } else {
            // piece p of S covers stages [p*nk/S, (p+1)*nk/S)
            const int j = (u - full) / S, piece = (u - full) % S;
            const int k0 = piece * nk / S;
            run_tau(full + j, k0, (piece + 1) * nk / S - k0,
                    parts + (size_t)(j * S + piece) * TP::PART_ELEMS, piece == 0 ? j : -1);
        }
    }
}

// The fragment rows of one (GEMM wave, fragment-row pair) of a tail tile
// cut into S pieces: each fragment's S pieces are loaded together and added
// in piece order, one fragment row at a time.
template <int MODE, class C, int S>
__device__ __forceinline__ void fixup_rows(__amdgpu_buffer_rsrc_t pres, int loff, int wave, int p,
                                           void *o, int64_t ldo, int m_valid, int n_valid) {
    static_assert(S >= 2 && S <= kSplitMaxPieces, "piece count");
    constexpr int NP = C::TN / 2;
#pragma unroll 1
    for (int m = 0; m < C::TM; ++m) {
        // fragment rows wholly past the valid edge: no partials were stored
        if ((wave >> 1) * C::WTM + m * 16 >= m_valid) break;
        floatx4 sum[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int f = wave * C::WAVE_BYTES + ((p + h * NP) * C::TM + m) * 1024;
            floatx4 v[S];
#pragma unroll
            for (int q = 0; q < S; ++q)
                v[q] = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(
                                                       pres, loff, q * C::PART_BYTES + f, 0));
            floatx4 r = v[0];
#pragma unroll
            for (int q = 1; q < S; ++q) {
                r[0] += v[q][0];
                r[1] += v[q][1];
                r[2] += v[q][2];
                r[3] += v[q][3];
            }
            sum[h] = r;
        }
        const int lane = threadIdx.x & 63;
        if (MODE == 0) {
            store_gateup<C>(sum[0], sum[1], p, m, wave & 1, wave >> 1, lane,
                            reinterpret_cast<bf16_t *>(o), ldo, m_valid, n_valid);
        } else {
            store_down<C>(sum[0], p, m, wave & 1, wave >> 1, lane, reinterpret_cast<float *>(o),
                          ldo, m_valid, n_valid);
            store_down<C>(sum[1], p + NP, m, wave & 1, wave >> 1, lane,
                          reinterpret_cast<float *>(o), ldo, m_valid, n_valid);
        }
    }
}

// Sum of the K pieces of the grouped GEMM's tail tiles, then the tile
// epilogue.  Work unit = (tail tile, GEMM wave), taken grid-stride by
// workgroups of four waves, one wave per fragment-row pair of that GEMM
// wave: it loads a fragment's S pieces together, adds them in piece order
// (p0 + p1 + ...), so the result is the same whichever piece finished first,
// and stores the pair as the GEMM's own epilogue would.  With no tail tiles
// (the host does not know the count) every workgroup returns at once.
template <int MODE, class TP>
__global__ __launch_bounds__(256) void split_fixup_kernel(const float *__restrict__ parts,
                                                         const int32_t *__restrict__ meta,
                                                         void *out, int64_t ldo) {
    using C = typename TP::C;
    constexpr int NP = C::TN / 2;  // fragment-row pairs per wave
    static_assert(NP * 64 == 256, "one wave per fragment-row pair");
    const int ntail = meta[0];
    const int S_eq = meta[1];  // equal pieces per tile, or 0: stream-K over P units
    const int P = meta[2], nk = meta[3];
    const int64_t W = (int64_t)ntail * nk;
    const int p = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    for (int unit = blockIdx.x; unit < ntail * 8; unit += gridDim.x) {
        const int j = unit / 8;
        const int wave = unit % 8;
        // the tile's pieces sit in consecutive slots [first, first + S), in K order
        int first, S;
        if (S_eq > 0) {
            first = j * S_eq;
            S = S_eq;
        } else {
            // units holding the tile's first and last stage (the unit of
            // stage s is the last u with u * W / P <= s)
            const int u0 = (int)((((int64_t)j * nk + 1) * P - 1) / W);
            const int u1 = (int)(((int64_t)(j + 1) * nk * P - 1) / W);
            first = u0 + j;
            S = u1 - u0 + 1;
        }
        const int32_t *md = meta + 4 + 4 * j;
        const int64_t r0 = md[0], n0 = md[1];
        const int m_valid = md[2], n_valid = md[3];
        const __amdgpu_buffer_rsrc_t pres = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(parts) + (size_t)first * C::PART_ELEMS, 0, -1, kBufferFlags);
        const int loff = lane * 16;
        void *o = MODE == 0 ? (void *)(reinterpret_cast<bf16_t *>(out) + r0 * ldo + n0)
                            : (void *)(reinterpret_cast<float *>(out) + r0 * ldo + n0);
        switch (S) {  // a static piece count: loads and sums stay unrolled
            case 2: fixup_rows<MODE, C, 2>(pres, loff, wave, p, o, ldo, m_valid, n_valid); break;
            case 3: fixup_rows<MODE, C, 3>(pres, loff, wave, p, o, ldo, m_valid, n_valid); break;
            case 4: fixup_rows<MODE, C, 4>(pres, loff, wave, p, o, ldo, m_valid, n_valid); break;
            case 5: fixup_rows<MODE, C, 5>(pres, loff, wave, p, o, ldo, m_valid, n_valid); break;
            case 6: fixup_rows<MODE, C, 6>(pres, loff, wave, p, o, ldo, m_valid, n_valid); break;
            case 7: fixup_rows<MODE, C, 7>(pres, loff, wave, p, o, ldo, m_valid, n_valid); break;
            case 8: fixup_rows<MODE, C, 8>(pres, loff, wave, p, o, ldo, m_valid, n_valid); break;
            default: break;
        }
    }
}

// Tile policy of each scheduler: the ping-pong tile, 256 weight rows by BM
// token rows.  The grouped launch knows its experts' host row counts or
// only a bound on them (the tokens); the launch-cost model picks its height
// (group_launch_rows) up to the smallest that holds that bound, with 320
// rows (fewest LDS bytes per MFMA) above 256; a dense launch knows its
// expert's rows and takes the height whose tile count fills the grid best
// (dense_tile_rows).
#ifndef MOE_GEMM_PINGPONG
#define MOE_GEMM_PINGPONG 1
#endif
#if MOE_GEMM_PINGPONG
constexpr int kTokenTile = 320;
template <int MODE, int BM = kTokenTile> using TileOf = PingPong<MODE, BM>;
#else
constexpr int kTokenTile = 256;
template <int MODE, int BM = kTokenTile> using TileOf = FourWave<MODE, 256, 256, 32, 4>;
#endif
template <int MODE> using GroupTile = TileOf<MODE>;

// ---------------------------------------------------------------------------
// Skinny down tile for decode-sized grouped launches: every expert of the
// launch has at most BM (16, 32 or 64) rows, so its down GEMM is one row of
// tiles that streams the expert's weights once.  A workgroup is one wave
// and owns SK_BN output columns (weight rows) by the expert's rows over the
// whole K range: no K split, no fixup.  Weight and act rows stream through
// a ring of LDS stages of SK_BK K by LDS-DMA, all but one stage ahead, the
// 16-byte chunks of each row XOR-placed as in the ping-pong tile.  The ring depth is chosen per
// launch (dynamic LDS): the deepest with which every tile of the launch is
// resident at once (a second, partial round of tiles would take as long as
// the first).  The MFMA (16x16x32 bf16, the weight fragment as the A
// operand, K ascending from 0) and the fragment contents are the ping-pong
// tile's, so the outputs carry the same bits as every other tile height in
// exact order.  The fragment reads and their wait are one assembly block:
// the compiler would otherwise wait for all LDS-DMA in flight before
// reading LDS and drain the ring every stage.
constexpr int SK_BN = 64;  // weight rows (output columns) per tile
// K per ring stage: 64, so each stage reads 128 contiguous bytes of every
// weight row.  With 32 (64-byte pieces of rows 3-12 KB apart) the weight
// stream ran 13-27% slower, even where the wider stages leave fewer tiles
// resident per compute unit.
constexpr int SK_BK = 64;
constexpr int SK_NS_MAX = 16;             // ring stages at most
constexpr size_t SK_LDS_MAX = 64 * 1024;  // dynamic LDS of one workgroup at most

// stages a wave can keep ahead: vmcnt counts at most 63 requests
constexpr int sk_ahead_max(int lps) { return std::min(SK_NS_MAX - 1, 63 / lps); }
// LDS-DMA requests per stage (64 lanes x 16 bytes each)
constexpr int sk_lps(int bm, int bk) { return (SK_BN + bm) * bk * 2 / 1024; }

// LDS bytes of a workgroup with a ring of ns stages of bk K: the ring plus
// room for the act-fragment reads a tile of fewer than 64 rows does not use
constexpr size_t sk_lds_bytes(int bm, int bk, int ns) {
    return (size_t)ns * (SK_BN + bm) * bk * 2 + (size_t)(4 - bm / 16) * 16 * bk * 2;
}

// one K-step's fragments: 4 weight fragments from wa, 4 act fragments from
// xa (a tile of fewer rows reads the first ones; the others land in the
// next slot or the padding after the ring), F bytes (16 LDS rows) apart
template <int F>
__device__ __forceinline__ void sk_read_frags(bf16x8 (&f)[8], uint32_t wa, uint32_t xa) {
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %8 offset:%10\n\t"
        "ds_read_b128 %2, %8 offset:%11\n\t"
        "ds_read_b128 %3, %8 offset:%12\n\t"
        "ds_read_b128 %4, %9\n\t"
        "ds_read_b128 %5, %9 offset:%10\n\t"
        "ds_read_b128 %6, %9 offset:%11\n\t"
        "ds_read_b128 %7, %9 offset:%12\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(f[0]), "=&v"(f[1]), "=&v"(f[2]), "=&v"(f[3]), "=&v"(f[4]), "=&v"(f[5]),
          "=&v"(f[6]), "=&v"(f[7])
        : "v"(wa), "v"(xa), "i"(F), "i"(2 * F), "i"(3 * F)
        : "memory");
}

// s_waitcnt vmcnt(LPS * n), 0 <= n <= K
template <int LPS, int K = sk_ahead_max(LPS)>
__device__ __forceinline__ void sk_wait(int n) {
    if (n == K) {
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(K * LPS) : "memory");
    } else if constexpr (K > 0) {
        sk_wait<LPS, K - 1>(n);
    }
}

// y[r0 + r][n0 .. n0 + 63] = w_down[e_first + e][n0 ..] . act[r0 + r] for
// the r < rows of expert e (offsets indexed by e_first + e, as in the other
// launches); grid = e_count * (N / SK_BN), ns ring stages of BK K.
template <int BM, int BK>
__global__ __launch_bounds__(64) void skinny_down_kernel(const int32_t *__restrict__ offsets,
                                                         int e_first, int e_count,
                                                         const bf16_t *__restrict__ act,
                                                         const bf16_t *__restrict__ w,
                                                         int64_t wstride, int N, int K,
                                                         float *__restrict__ y, int ns) {
    constexpr int TN = SK_BN / 16, TM = BM / 16;
    static_assert(TM <= 4, "at most 4 act fragments per K-step");
    static_assert(BK == 32 || BK == 64, "16-byte chunks: 4 or 8 per LDS row");
    constexpr int CPR = BK / 8;    // 16-byte chunks per LDS row
    constexpr int RPI = 64 / CPR;  // rows one LDS-DMA request fills
    constexpr int WI = SK_BN / RPI, XI = BM / RPI;
    constexpr int LPS = WI + XI;
    static_assert(LPS == sk_lps(BM, BK), "requests per stage");
    constexpr int STAGE = (SK_BN + BM) * BK;  // bf16 elements
    constexpr int F = 16 * BK * 2;            // bytes of 16 LDS rows
    constexpr int KH = BK / 32;               // MFMA K-steps per stage
    // ring of ns stages (2 <= ns <= sk_ahead_max(LPS) + 1), sk_lds_bytes
    extern __shared__ __attribute__((aligned(16))) bf16_t smem[];

    const int NT = N / SK_BN;
    const int e = blockIdx.x / NT;
    const int nt = blockIdx.x - e * NT;
    if (e >= e_count) return;
    const int r0 = offsets[e_first + e];
    const int rows = offsets[e_first + e + 1] - r0;  // <= BM (the launcher's bound)
    if (rows <= 0) return;
    const int lane = threadIdx.x;
    const int64_t n0 = (int64_t)nt * SK_BN;

    // LDS-DMA sources: lane i fetches row (i / CPR) of an RPI-row request,
    // the 16-byte chunk (i % CPR) ^ swz(row) of the stage's BK K, into
    // place i % CPR
    const int drow = lane / CPR;
    const int dchunk = ((lane % CPR) ^ swz<BK>(drow)) * 8;
    const bf16_t *src[LPS];
    const bf16_t *we = w + (int64_t)(e_first + e) * wstride;
#pragma unroll
    for (int i = 0; i < WI; ++i) src[i] = we + (n0 + i * RPI + drow) * K + dchunk;
#pragma unroll
    for (int i = 0; i < XI; ++i) {
        const int j = min(i * RPI + drow, rows - 1);  // rows past the expert's: repeats
        src[WI + i] = act + (int64_t)(r0 + j) * K + dchunk;
    }
    const int nk = K / BK;
    auto issue = [&](int kt, int slot) {
        bf16_t *sb = smem + slot * STAGE;
#pragma unroll
        for (int i = 0; i < LPS; ++i)
            __builtin_amdgcn_global_load_lds((gbl_void_t *)(src[i] + kt * BK),
                                             (lds_void_t *)(sb + i * RPI * BK), 16, 0, 0);
    };

    // fragment addresses in ring slot 0, K-step h of the stage: weight row
    // t * 16 + lrow and act row m * 16 + lrow, the chunk holding K
    // 32 h + 8 (lane / 16) .. + 7
    const int lrow = lane & 15;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void_t *)smem;
    uint32_t wa0[KH], xa0[KH];
#pragma unroll
    for (int h = 0; h < KH; ++h) {
        const int chunk = ((h * 4 + (lane >> 4)) ^ swz<BK>(lrow)) * 8;
        wa0[h] = lds0 + (uint32_t)((lrow * BK + chunk) * 2);
        xa0[h] = wa0[h] + (uint32_t)(SK_BN * BK * 2);
    }

    floatx4 acc[TN][TM];
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
        for (int m = 0; m < TM; ++m) acc[t][m] = floatx4{0.f, 0.f, 0.f, 0.f};

    // stage kt goes to ring slot kt % ns
    const int ahead = ns - 1;
    for (int kt = 0; kt < min(ahead, nk); ++kt) issue(kt, kt);
    int wslot = ahead, rslot = 0;  // slots of stages kt + ahead and kt
    for (int kt = 0; kt < nk; ++kt) {
        // stage kt + ahead into the slot read at kt - 1
        if (kt + ahead < nk) issue(kt + ahead, wslot);
        wslot = wslot + 1 == ns ? 0 : wslot + 1;
        sk_wait<LPS>(min(ahead, nk - 1 - kt));  // stage kt landed
        const uint32_t so = (uint32_t)(rslot * STAGE * 2);
        rslot = rslot + 1 == ns ? 0 : rslot + 1;
#pragma unroll
        for (int h = 0; h < KH; ++h) {
            bf16x8 f[8];
            sk_read_frags<F>(f, wa0[h] + so, xa0[h] + so);
#pragma unroll
            for (int m = 0; m < TM; ++m)
#pragma unroll
                for (int t = 0; t < TN; ++t)
                    acc[t][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f[t], f[4 + m],
                                                                        acc[t][m], 0, 0, 0);
        }
    }

    // epilogue: the lane holds output columns t * 16 + 4 (lane / 16) .. + 3
    // of row m * 16 + (lane % 16)
    const int ocol = (lane >> 4) * 4;
#pragma unroll
    for (int m = 0; m < TM; ++m) {
        const int row = m * 16 + lrow;
        if (row >= rows) continue;
        float *o = y + (int64_t)(r0 + row) * N + n0;
#pragma unroll
        for (int t = 0; t < TN; ++t) *reinterpret_cast<floatx4 *>(o + t * 16 + ocol) = acc[t][m];
    }
}

// Ring depth of a launch of `tiles` non-empty tiles: the deepest ring (at
// most sk_ahead_max + 1 stages, SK_LDS_MAX bytes) with which the tiles of a
// compute unit all fit its LDS at once, and at least 4 stages.
int sk_ring(int bm, int bk, int64_t tiles) {
    const int cus = device_cu_count();
    const int64_t per_cu = std::max<int64_t>(1, (tiles + cus - 1) / cus);
    const size_t cap = std::min<size_t>(SK_LDS_MAX, (size_t)(160 * 1024) / per_cu);
    int ns = sk_ahead_max(sk_lps(bm, bk)) + 1;
    while (ns > 4 && sk_lds_bytes(bm, bk, ns) > cap) --ns;
    return ns;
}

template <int BM, int BK>
hipError_t skinny_down_launch(unsigned blocks, int64_t tiles, const int32_t *offsets,
                              int e_first, int e_count, const bf16_t *act, const bf16_t *w,
                              int64_t wstride, int N, int K, float *y, hipStream_t s) {
    if (K % BK) return hipErrorInvalidValue;
    const int ns = sk_ring(BM, BK, tiles);
    if (ns < 2 || ns - 1 > sk_ahead_max(sk_lps(BM, BK)) || sk_lds_bytes(BM, BK, ns) > SK_LDS_MAX)
        return hipErrorInvalidValue;
    skinny_down_kernel<BM, BK><<<blocks, 64, sk_lds_bytes(BM, BK, ns), s>>>(
        offsets, e_first, e_count, act, w, wstride, N, K, y, ns);
    return hipGetLastError();
}

int round_grid(int64_t tiles) { return (int)(((tiles + NXCD - 1) / NXCD) * NXCD); }

// Fixup launch after a grouped GEMM that was given a split buffer: fewer
// than grid tail tiles can be cut (each into two or more pieces), 8 work
// units each; one workgroup per compute unit at most, so an empty fixup is
// cheap to dispatch.
template <int MODE, class TP>
hipError_t launch_split_fixup(int grid, const float *parts, const int32_t *meta, void *out,
                              int64_t ldo, hipStream_t s) {
    if constexpr (!TP::CAN_SPLIT) {
        return hipSuccess;
    } else {
        const int max_tail = std::min(grid, kSplitMaxTail);
        const int blocks = std::min(max_tail * 8, device_cu_count());
        split_fixup_kernel<MODE, TP><<<blocks, 256, 0, s>>>(parts, meta, out, ldo);
        return hipGetLastError();
    }
}

template <int MODE, class TP>
hipError_t group_launch(const int32_t *offsets, int e_first, int e_count, const bf16_t *x,
                        const int32_t *row_map, int slot_div, const bf16_t *w0s,
                        const bf16_t *w1s, int64_t wstride, int N, int K, void *out,
                        int64_t ldo, int grid, float *parts, int32_t *split_meta, int rows_one,
                        hipStream_t s) {
    const bool split = parts != nullptr && split_meta != nullptr;
    group_kernel<MODE, TP><<<grid, TP::THREADS, 0, s>>>(
        offsets, e_first, e_count, x, row_map, slot_div, w0s, w1s, wstride, N, K, out, ldo,
        split ? parts : nullptr, split ? split_meta : nullptr, rows_one);
    if (split) return launch_split_fixup<MODE, TP>(grid, parts, split_meta, out, ldo, s);
    return hipGetLastError();
}

template <int MODE>
hipError_t group_launch_bm(int bm, const int32_t *offsets, int e_first, int e_count,
                           const bf16_t *x, const int32_t *row_map, int slot_div,
                           const bf16_t *w0s, const bf16_t *w1s, int64_t wstride, int N, int K,
                           void *out, int64_t ldo, int grid, float *parts, int32_t *split_meta,
                           int rows_one, hipStream_t s) {
#define MOE_GROUP_LAUNCH(BMV)                                                                   \
    return group_launch<MODE, TileOf<MODE, BMV>>(offsets, e_first, e_count, x, row_map,       \
                                                 slot_div, w0s, w1s, wstride, N, K, out, ldo, \
                                                 grid, parts, split_meta, rows_one, s)
#if MOE_GEMM_PINGPONG
    switch (bm) {
        case 128: MOE_GROUP_LAUNCH(128);
        case 192: MOE_GROUP_LAUNCH(192);
        case 256: MOE_GROUP_LAUNCH(256);
        default: MOE_GROUP_LAUNCH(320);
    }
#else
    MOE_GROUP_LAUNCH(256);
#endif
#undef MOE_GROUP_LAUNCH
}

template <int MODE, class TP>
hipError_t dense_launch(int64_t rows, const bf16_t *x, const bf16_t *w0, const bf16_t *w1, int N,
                        int K, void *out, int64_t ldo, hipStream_t s) {
    const int MT = (int)((rows + TP::BM - 1) / TP::BM);
    const int NT = (N + TP::BNOUT - 1) / TP::BNOUT;
    dense_kernel<MODE, TP><<<round_grid((int64_t)MT * NT), TP::THREADS, 0, s>>>(
        x, rows, w0, w1, N, K, out, ldo, MT, NT);
    return hipGetLastError();
}

template <int MODE>
hipError_t dense_launch_bm(int bm, int64_t rows, const bf16_t *x, const bf16_t *w0,
                           const bf16_t *w1, int N, int K, void *out, int64_t ldo, hipStream_t s) {
#if MOE_GEMM_PINGPONG
    switch (bm) {
        case 128: return dense_launch<MODE, TileOf<MODE, 128>>(rows, x, w0, w1, N, K, out, ldo, s);
        case 192: return dense_launch<MODE, TileOf<MODE, 192>>(rows, x, w0, w1, N, K, out, ldo, s);
        case 256: return dense_launch<MODE, TileOf<MODE, 256>>(rows, x, w0, w1, N, K, out, ldo, s);
        default: return dense_launch<MODE, TileOf<MODE, 320>>(rows, x, w0, w1, N, K, out, ldo, s);
    }
#else
    return dense_launch<MODE, TileOf<MODE>>(rows, x, w0, w1, N, K, out, ldo, s);
#endif
}

// ---- launch cost model (host) ---------------------------------------------
// Device time of one launch of the persistent scheduler, from per-tile costs
// of each tile height measured on MI355X (microseconds):
//   tile time = K / 32 * step(MODE, BM) + epi(MODE, BM)
// (step: the cost of 32 K, whatever the tile's stage depth).  Tiles run in rounds of G
// workgroups; a partial round of rem tiles takes the fraction
// kPartialRound[MODE] + (1 - kPartialRound) * busy of a full round's K loop
// (busy = the fraction of workgroups with work: fewer active compute units
// run each tile faster), then the epilogue.  With the K split, a partial
// last round of rem <= G/2 tiles is cut into S pieces as the scheduler does
// (S = min(8, G/rem, stages/32, slots/rem)): its K loop is S times shorter, and
// the fixup costs a fixed time plus a time per partial-sum block (its bytes
// grow with BM).  Each launch pays a fixed start-up and drain time.
struct TileCost {
    int bm;
    double step_us[2];  // 32 K of a 256 x BM tile: gate/up, down
    double epi_us[2];   // a tile's epilogue: gate/up (bf16 SiLU*mul), down (fp32)
};
// Fitted by least squares (4.0% rms gate/up, 4.5% down, 14% worst) to one
// expert's dense launches at 512 .. 32768 rows on the DeepSeekV2 (H 5120,
// I 1536) and Mixtral (H 4096, I 3584) expert shapes, every tile height,
// with and without the K split (bench.py --tile-study).
constexpr TileCost kTileCosts[] = {
    {320, {0.896, 1.004}, {13.0, 12.3}},
    {256, {0.750, 0.839}, {14.6, 12.8}},
    {192, {0.607, 0.715}, {10.7, 9.3}},
    {128, {0.441, 0.471}, {6.2, 7.7}},
};
constexpr double kLaunchUs[2] = {12.9, 6.4};     // start-up + drain: gate/up, down
constexpr double kPartialRound[2] = {0.69, 0.71};
constexpr double kFixupUs[2] = {0.0, 2.3};       // fixup launch with work
constexpr double kFixupBlockUs[2] = {0.0994, 0.0864};  // per 256 x 320 partial block

const TileCost &tile_cost(int bm) {
    for (const TileCost &c : kTileCosts)
        if (c.bm == bm) return c;
    return kTileCosts[0];
}

}  // namespace

double gemm_launch_us(int mode, int bm, int64_t tiles, int K, int grid, bool split) {
    if (tiles <= 0) return 0.0;
    const TileCost &c = tile_cost(bm);
    const int md = mode ? 1 : 0;
    const double loop_us = K / 32 * c.step_us[md];
    const int nk = K / pp_stage_k(bm);  // the tile's K stages, as the kernel cuts them
    const int64_t full_rounds = tiles / grid;
    const int64_t rem = tiles % grid;
    double us = kLaunchUs[md] + full_rounds * (loop_us + c.epi_us[md]);
    if (rem > 0) {
        // (a round of more than half the grid that the kernel spreads
        // stream-K, for tall tiles at most half full, is priced unsplit: an
        // upper bound)
        int S = 1;
        if (split && 2 * rem <= grid) {
            S = (int)std::min<int64_t>(
                std::min<int64_t>(kSplitMaxPieces, grid / rem),
                std::min<int64_t>(nk / (full_rounds == 0 ? kSplitMinStagesAlone : kSplitMinStages),
                                  kSplitSlots / rem));
        }
        const double busy = (double)std::min<int64_t>(grid, rem * std::max(S, 1)) / grid;
        const double part = kPartialRound[md] + (1.0 - kPartialRound[md]) * busy;
        if (S >= 2)
            us += loop_us / S * part + c.epi_us[md] + kFixupUs[md] +
                  kFixupBlockUs[md] * (double)(rem * S) * bm / 320.0;
        else
            us += loop_us * part + c.epi_us[md];
    }
    return us;
}

int64_t gemm_tiles(int mode, int bm, int64_t rows, int N) {
    const int bnout = mode == 0 ? 128 : 256;
    return ((rows + bm - 1) / bm) * ((N + bnout - 1) / bnout);
}

double ffn_expert_us(int bm, int64_t rows, int H, int I, int grid, bool split) {
    return gemm_launch_us(0, bm, gemm_tiles(0, bm, rows, I), H, grid, split) +
           gemm_launch_us(1, bm, gemm_tiles(1, bm, rows, H), I, grid, split);
}

int dense_tile_rows(int64_t rows, int H, int I, int grid, bool split) {
#if MOE_GEMM_PINGPONG
    int best = kTokenTile;
    double best_us = 0.0;
    for (const TileCost &c : kTileCosts) {
        const double us = ffn_expert_us(c.bm, rows, H, I, grid, split);
        if (best_us == 0.0 || us < best_us) {
            best = c.bm;
            best_us = us;
        }
    }
    return best;
#else
    return kTokenTile;
#endif
}

int group_tile_rows(int64_t max_rows) {
#if MOE_GEMM_PINGPONG
    // below the tallest tile, the smallest height that still holds every
    // expert's rows in one tile: fewer padded rows, never more tiles
    if (max_rows <= 128) return 128;
    if (max_rows <= 192) return 192;
    if (max_rows <= 256) return 256;
#endif
    (void)max_rows;
    return kTokenTile;
}

namespace {

constexpr int kTileHeights[4] = {128, 192, 256, 320};

// Expected m-tiles of one expert for each tile height, E[ceil(min(r, cap)
// / bm)], where its row count r ~ Binomial(tokens, p): every token picks
// the expert with probability p (top_k distinct of E experts, uniform).
// The probabilities are walked out from the mode by the ratio of
// neighbouring terms until they fall below 1e-12 of the mode's.
void expected_mtiles(int64_t tokens, double p, int64_t cap, double out[4]) {
    for (int i = 0; i < 4; ++i) out[i] = 0.0;
    if (tokens <= 0 || cap <= 0 || p <= 0.0) return;
    auto add = [&](int64_t r, double pr) {
        const int64_t rr = std::min(r, cap);
        for (int i = 0; i < 4; ++i) out[i] += pr * (double)((rr + kTileHeights[i] - 1) / kTileHeights[i]);
    };
    if (p >= 1.0) {
        add(tokens, 1.0);
        return;
    }
    const double q = 1.0 - p, n = (double)tokens;
    const int64_t mode = std::min<int64_t>(tokens, (int64_t)((n + 1.0) * p));
    const double m = (double)mode;
    const double pm = std::exp(std::lgamma(n + 1.0) - std::lgamma(m + 1.0) -
                               std::lgamma(n - m + 1.0) + m * std::log(p) + (n - m) * std::log(q));
    double total = pm, pr = pm;
    add(mode, pm);
    for (int64_t r = mode; r < tokens; ++r) {
        pr *= (double)(tokens - r) / (double)(r + 1) * (p / q);
        if (pr < 1e-12 * pm) break;
        add(r + 1, pr);
        total += pr;
    }
    pr = pm;
    for (int64_t r = mode; r > 0; --r) {
        pr *= (double)r / (double)(tokens - r + 1) * (q / p);
        if (pr < 1e-12 * pm) break;
        add(r - 1, pr);
        total += pr;
    }
    for (int i = 0; i < 4; ++i) out[i] /= total;
}

}  // namespace

int group_launch_rows(int64_t max_rows, const int32_t *rows, int n_experts, int64_t tokens,
                      double p, int H, int I, int grid, bool split) {
    const int cap = group_tile_rows(max_rows);
#if MOE_GEMM_PINGPONG
    if (n_experts <= 0 || cap == kTileHeights[0]) return cap;
    double mt[4];
    if (rows == nullptr) expected_mtiles(tokens, p, max_rows, mt);
    double us[4] = {0.0, 0.0, 0.0, 0.0};
    int best = -1, icap = 0;
    for (int i = 0; i < 4 && kTileHeights[i] <= cap; ++i) {
        const int bm = kTileHeights[i];
        int64_t tiles_gu = 0, tiles_dn = 0;
        if (rows != nullptr) {
            for (int e = 0; e < n_experts; ++e) {
                tiles_gu += gemm_tiles(0, bm, rows[e], I);
                tiles_dn += gemm_tiles(1, bm, rows[e], H);
            }
        } else {
            const double m = n_experts * mt[i];
            tiles_gu = std::llround(m * (double)gemm_tiles(0, bm, bm, I));
            tiles_dn = std::llround(m * (double)gemm_tiles(1, bm, bm, H));
        }
        us[i] = gemm_launch_us(0, bm, tiles_gu, H, grid, split) +
                gemm_launch_us(1, bm, tiles_dn, I, grid, split);
        if (best < 0 || us[i] < us[best]) best = i;
        icap = i;
    }
    // another height only for a predicted gain above the model's error
    return us[best] < (1.0 - kGroupRowsMinGain) * us[icap] ? kTileHeights[best] : cap;
#else
    (void)rows, (void)n_experts, (void)tokens, (void)p, (void)H, (void)I, (void)grid, (void)split;
    return cap;
#endif
}

bool valid_tile_rows(int bm) {
#if MOE_GEMM_PINGPONG
    return bm == 128 || bm == 192 || bm == 256 || bm == 320;
#else
    return bm == kTokenTile;
#endif
}

hipError_t launch_dense_gateup(int64_t rows, int H, int I, const bf16_t *x, const bf16_t *w_gate,
                               const bf16_t *w_up, bf16_t *act, int bm, hipStream_t s) {
    if (rows <= 0) return hipSuccess;
    return dense_launch_bm<0>(bm, rows, x, w_gate, w_up, I, H, act, I, s);
}

hipError_t launch_dense_down(int64_t rows, int H, int I, const bf16_t *act,
                             const bf16_t *w_down, float *y, int bm, hipStream_t s) {
    if (rows <= 0) return hipSuccess;
    return dense_launch_bm<1>(bm, rows, act, w_down, nullptr, H, I, y, H, s);
}

size_t gemm_split_bytes() {
    // the tallest tile has the largest block of partial sums
    const size_t e = std::max(GroupTile<0>::PART_ELEMS, GroupTile<1>::PART_ELEMS);
    return e * sizeof(float) * kSplitSlots;
}

hipError_t launch_group_gateup(const moe_dims &d, int e_first, int e_count,
                               const int32_t *offsets, const bf16_t *x_rows,
                               const int32_t *row_map, const bf16_t *w_gate,
                               const bf16_t *w_up, bf16_t *act, int grid, float *parts,
                               int32_t *split_meta, int bm, hipStream_t s, int64_t rows_one) {
    if (e_count <= 0) return hipSuccess;
    if (!offsets && (e_count != 1 || rows_one < 0 || rows_one > INT32_MAX))
        return hipErrorInvalidValue;
    return group_launch_bm<0>(bm, offsets, e_first, e_count, x_rows, row_map, d.top_k, w_gate,
                              w_up, (int64_t)d.inter * d.hidden, d.inter, d.hidden, act,
                              d.inter, grid, parts, split_meta, (int)rows_one, s);
}

hipError_t launch_group_down(const moe_dims &d, int e_first, int e_count,
                             const int32_t *offsets, const bf16_t *act,
                             const bf16_t *w_down, float *y_perm, int grid, float *parts,
                             int32_t *split_meta, int bm, hipStream_t s, int64_t rows_one) {
    if (e_count <= 0) return hipSuccess;
    if (!offsets && (e_count != 1 || rows_one < 0 || rows_one > INT32_MAX))
        return hipErrorInvalidValue;
    return group_launch_bm<1>(bm, offsets, e_first, e_count, act, nullptr, 1, w_down, nullptr,
                              (int64_t)d.hidden * d.inter, d.hidden, d.inter, y_perm, d.hidden,
                              grid, parts, split_meta, (int)rows_one, s);
}

int skinny_down_rows(int64_t max_rows, int64_t active_experts, int N) {
    if (max_rows > kSkinnyMaxRows || N % SK_BN) return 0;
    if (active_experts * (N / SK_BN) < 2 * (int64_t)device_cu_count()) return 0;
    return max_rows <= 16 ? 16 : max_rows <= 32 ? 32 : 64;
}

hipError_t launch_skinny_down(const moe_dims &d, int e_first, int e_count,
                              const int32_t *offsets, const bf16_t *act, const bf16_t *w_down,
                              float *y_perm, int bm, int64_t active_experts, hipStream_t s) {
    if (e_count <= 0) return hipSuccess;
    const int N = d.hidden, K = d.inter;
    if (N % SK_BN || K % SK_BK) return hipErrorInvalidValue;
    const unsigned blocks = (unsigned)(e_count * (N / SK_BN));
    const int64_t active = std::min<int64_t>(e_count, std::max<int64_t>(1, active_experts));
    const int64_t tiles = active * (N / SK_BN);
    const int64_t wstride = (int64_t)N * K;
    switch (bm) {
        case 16:
            return skinny_down_launch<16, SK_BK>(blocks, tiles, offsets, e_first, e_count, act,
                                                 w_down, wstride, N, K, y_perm, s);
        case 32:
            return skinny_down_launch<32, SK_BK>(blocks, tiles, offsets, e_first, e_count, act,
                                                 w_down, wstride, N, K, y_perm, s);
        case 64:
            return skinny_down_launch<64, SK_BK>(blocks, tiles, offsets, e_first, e_count, act,
                                                 w_down, wstride, N, K, y_perm, s);
        default:
            return hipErrorInvalidValue;
    }
}

}  // namespace moe
