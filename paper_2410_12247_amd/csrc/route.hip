// Router: fp32 logits, top-k selection and softmax weights in one kernel.
//
// Logits (the topKGating operator): every logit is ONE fp32 fma chain over
// h in ascending order, started from +0, with the bias added once at the
// end -- the same bits as a sequential fma loop on the CPU.  A thread keeps
// a 4-token x TE-expert block of chains in registers; x and the router are
// staged through LDS 32 h at a time.
//
// Selection: the token's logits are spread over a wave (lane l holds experts
// l, l+64, l+128, l+192); each of the k rounds is a wave-wide max of 64-bit
// keys (order-preserving logit bits << 32 | inverted expert index, so ties
// go to the lower index) built from DPP row permutes and readlane.  The
// winner's lane clears its key.  Softmax weights are computed in fp64 and
// rounded to fp32 once; the full-softmax denominator is a DPP wave sum.
#include "common.h"

#include <type_traits>

#include "route_lane_asm.h"

namespace moe {
namespace {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

constexpr int RT_THREADS = 256;

template <int CTRL>
__device__ __forceinline__ uint32_t dpp32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, 0xF, 0xF, false);
}

__device__ __forceinline__ uint64_t max_u64(uint64_t a, uint64_t b) { return a > b ? a : b; }

template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
    uint32_t lo = dpp32<CTRL>((uint32_t)v);
    uint32_t hi = dpp32<CTRL>((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
    uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

// Wave-wide max: butterfly inside each 16-lane row (quad_perm 1032, quad_perm
// 2301, half-row mirror, row mirror), then the four row results by readlane.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t k) {
    k = max_u64(k, dpp64<0xB1>(k));
    k = max_u64(k, dpp64<0x4E>(k));
    k = max_u64(k, dpp64<0x141>(k));
    k = max_u64(k, dpp64<0x140>(k));
    return max_u64(max_u64(readlane64(k, 0), readlane64(k, 16)),
                   max_u64(readlane64(k, 32), readlane64(k, 48)));
}

__device__ __forceinline__ double dpp_f64(double v, int which) {
    uint64_t b = __builtin_bit_cast(uint64_t, v);
    uint64_t r;
    switch (which) {
        case 0: r = dpp64<0xB1>(b); break;
        case 1: r = dpp64<0x4E>(b); break;
        case 2: r = dpp64<0x141>(b); break;
        default: r = dpp64<0x140>(b); break;
    }
    return __builtin_bit_cast(double, r);
}

// Wave-wide fp64 sum; every lane combines the same pairs (commutative adds),
// so the result is identical in all lanes and from run to run.
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v = v + dpp_f64(v, i);
    uint64_t b = __builtin_bit_cast(uint64_t, v);
    double r0 = __builtin_bit_cast(double, readlane64(b, 0));
    double r1 = __builtin_bit_cast(double, readlane64(b, 16));
    double r2 = __builtin_bit_cast(double, readlane64(b, 32));
    double r3 = __builtin_bit_cast(double, readlane64(b, 48));
    return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ uint64_t logit_key(float z, int e) {
    uint32_t u = __float_as_uint(z);
    if (u == 0x80000000u) u = 0;  // -0 ranks equal to +0
    const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)ord << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)e);
}

__device__ __forceinline__ float key_logit(uint64_t key) {
    const uint32_t ord = (uint32_t)(key >> 32);
    const uint32_t u = (ord & 0x80000000u) ? (ord & 0x7FFFFFFFu) : ~ord;
    return __uint_as_float(u);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Top-k and softmax weights of token t from its E logits (zrow, in LDS),
// by one wave: lane l holds experts l, l+64, l+128, l+192; each of the k
// rounds takes the wave-wide max key; the weights are fp64 softmax values
// rounded once to fp32.
__device__ __forceinline__ void select_token(const float *zrow, int64_t t, int E, int k,
                                             int renorm, int lane, int32_t *__restrict__ ids,
                                             float *__restrict__ wout) {
    uint64_t key[4];
    float zl[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane + 64 * q;
        zl[q] = e < E ? zrow[e] : 0.0f;
        key[q] = e < E ? logit_key(zl[q], e) : 0ull;
    }
    int sel_e[kMaxTopK];
    float sel_z[kMaxTopK];
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
        sel_e[j] = 0;
        sel_z[j] = 0.0f;
        if (j < k) {
            const uint64_t best =
                wave_max_u64(max_u64(max_u64(key[0], key[1]), max_u64(key[2], key[3])));
            sel_e[j] = (int)(0xFFFFFFFFu - (uint32_t)best);
            sel_z[j] = key_logit(best);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (key[q] == best) key[q] = 0ull;
        }
    }
    const double zmax = (double)sel_z[0];
    double denom;
    if (renorm) {
        denom = 0.0;
#pragma unroll
        for (int j = 0; j < kMaxTopK; ++j)
            if (j < k) denom += exp((double)sel_z[j] - zmax);
    } else {
        double part = 0.0;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (lane + 64 * q < E) part += exp((double)zl[q] - zmax);
        denom = wave_sum_f64(part);
    }
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
        if (j < k && lane == j) {
            ids[t * k + j] = sel_e[j];
            wout[t * k + j] = (float)(exp((double)sel_z[j] - zmax) / denom);
        }
    }
}

// One 16-byte-per-lane LDS-DMA request (lane l's bytes land at lds_addr +
// 16 l; lds_addr must be the same in every lane), written out so that the
// compiler does not see an LDS write in
// flight: it would put a full vmcnt(0) in front of every later LDS read,
// which makes the next chunk's loads finish before the current chunk is
// multiplied.  The kernel's own vmcnt wait and barrier order the data.
__device__ __forceinline__ void dma16_to_lds(const void *gptr, uint32_t lds_addr) {
    // the LDS address goes in through an "{m0}" operand, so the compiler
    // itself writes m0 (and knows it does); the s_nop separates that write
    // from the load that reads it
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gptr), "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

// Register-tiled router for more than 16 experts.
//
// Logits phase layout: 256 threads = TG token groups x EG expert groups
// (EG = 16, or 32 for 129 to 160 experts); a thread
// owns TT tokens (tg + TG i: consecutive lanes read rows 36 floats apart, so
// eight lanes of a 16-byte LDS read land on distinct banks) x TE experts
// (TE = ceil(E / EG)) and keeps their fma chains in registers.  x and the
// router are staged through two LDS buffers HC h at a time: the router rows
// by LDS-DMA, x through registers (widened to fp32), the next chunk in
// flight while the current one is multiplied; per 4 h a thread reads
// TT + TE float4 and issues 4*TT*TE fmas.
//
// TT tokens per thread, so a workgroup routes TG*TT <= 64 tokens; the
// launcher picks TT so that the grid keeps several workgroups per compute
// unit.
template <int TE, int TT, int RT_EG, int HC>
__global__ __launch_bounds__(RT_THREADS) void route_kernel(const bf16_t *__restrict__ x,
                                                           const float *__restrict__ wr,
                                                           const float *__restrict__ bias,
                                                           int64_t T, int H, int E, int k,
                                                           int renorm, int32_t *__restrict__ ids,
                                                           float *__restrict__ wout) {
    constexpr int RT_TG = RT_THREADS / RT_EG;  // token groups
    constexpr int RT_TOK = RT_TG * TT;          // tokens per workgroup
    static_assert(RT_TOK <= 64, "a workgroup routes at most 64 tokens");
    static_assert(HC % 32 == 0, "router rows are staged in 128-byte segments");
    constexpr int RT_TT = TT;
    constexpr int RT_HC = HC;
    constexpr int RT_LD = HC + 4;       // x row stride in LDS (floats)
    constexpr int EMAX = RT_EG * TE;
    constexpr int XS = RT_TOK * RT_LD;  // floats of one x stage
    constexpr int WS = EMAX * RT_HC;    // floats of one router stage
    constexpr int P1 = 2 * XS + 2 * WS;
    constexpr int P2 = RT_TOK * (EMAX + 1);  // selection phase
    __shared__ __attribute__((aligned(16))) float lds[P1 > P2 ? P1 : P2];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tg = tid % RT_TG;  // tokens tg + RT_TG*i, i < TT
    const int eg = tid / RT_TG;  // experts eg*TE .. +TE
    const int64_t t0 = (int64_t)blockIdx.x * RT_TOK;

    float acc[RT_TT][TE];
#pragma unroll
    for (int i = 0; i < RT_TT; ++i)
#pragma unroll
        for (int j = 0; j < TE; ++j) acc[i][j] = 0.0f;

    // x: 16-byte (8 bf16) pieces, PPT per thread, widened to fp32 in LDS;
    // piece p covers token row p / PPR, h 8 * (p % PPR) of the chunk
    constexpr int PPR = HC / 8;
    constexpr int NPIECE = RT_TOK * PPR;
    constexpr int PPT = (NPIECE + RT_THREADS - 1) / RT_THREADS;
    const bf16_t *xsrc[PPT];
    int xdst[PPT];
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
        const int pc = min(tid + RT_THREADS * q, NPIECE - 1);  // repeats write equal values
        const int64_t xt = min<int64_t>(t0 + pc / PPR, T - 1);
        xsrc[q] = x + xt * H + (pc % PPR) * 8;
        xdst[q] = (pc / PPR) * RT_LD + (pc % PPR) * 8;
    }
    // router: LDS-DMA of 8 rows x one 128-byte segment per wave-wide
    // instruction; stage layout [row block of 8][segment][8 rows][32 floats],
    // 16-byte chunk c of a row's segment at chunk c ^ (row & 7)
    constexpr int NSEG = HC / 32;
    const int n_wdma = (E + 7) / 8 * NSEG;
    const int drow = lane >> 3;
    const int dchunk = (lane & 7) ^ (drow & 7);
    auto issue_w = [&](int h0, float *wsb) {
        for (int q = wave; q < n_wdma; q += RT_THREADS / 64) {
            const int blk = q / NSEG, seg = q % NSEG;
            const int r = min(blk * 8 + drow, E - 1);  // rows past E: a copy, never read
            dma16_to_lds(wr + (int64_t)r * H + h0 + seg * 32 + dchunk * 4,
                         (uint32_t)(uintptr_t)(lds_void_t *)(wsb + blk * 8 * HC + seg * 256));
        }
    };

    uint4 xr[PPT];
#pragma unroll
    for (int q = 0; q < PPT; ++q) xr[q] = *reinterpret_cast<const uint4 *>(xsrc[q]);
    issue_w(0, lds + 2 * XS);
    const int nchunk = H / RT_HC;
    for (int c = 0; c < nchunk; ++c) {
        const int st = c & 1;
        float *xs = lds + st * XS;
        const float *ws = lds + 2 * XS + st * WS;
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const uint4 v = xr[q];
            const float4 a = make_float4(bf16_lo(v.x), bf16_hi(v.x), bf16_lo(v.y), bf16_hi(v.y));
            const float4 b = make_float4(bf16_lo(v.z), bf16_hi(v.z), bf16_lo(v.w), bf16_hi(v.w));
            *reinterpret_cast<float4 *>(xs + xdst[q]) = a;
            *reinterpret_cast<float4 *>(xs + xdst[q] + 4) = b;
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this chunk's router rows landed
        __syncthreads();  // ... for every wave; chunk c-1 fully consumed
        if (c + 1 < nchunk) {
#pragma unroll
            for (int q = 0; q < PPT; ++q)
                xr[q] = *reinterpret_cast<const uint4 *>(xsrc[q] + (c + 1) * RT_HC);
            issue_w((c + 1) * RT_HC, lds + 2 * XS + (st ^ 1) * WS);
        }
#pragma unroll
        for (int hh = 0; hh < RT_HC; hh += 4) {
            // all operands of this 4-h step first, then the fmas
            float4 xv[RT_TT], wv[TE];
#pragma unroll
            for (int i = 0; i < RT_TT; ++i)
                xv[i] = *reinterpret_cast<const float4 *>(xs + (tg + RT_TG * i) * RT_LD + hh);
#pragma unroll
            for (int j = 0; j < TE; ++j) {
                const int e = min(eg * TE + j, EMAX - 1);
                wv[j] = *reinterpret_cast<const float4 *>(
                    ws + (e >> 3) * 8 * HC + (hh >> 5) * 256 + (e & 7) * 32 +
                    ((((hh >> 2) & 7) ^ (e & 7)) << 2));
            }
#pragma unroll
            for (int j = 0; j < TE; ++j) {
#pragma unroll
                for (int i = 0; i < RT_TT; ++i) {
                    float v = acc[i][j];
                    v = __builtin_fmaf(xv[i].x, wv[j].x, v);
                    v = __builtin_fmaf(xv[i].y, wv[j].y, v);
                    v = __builtin_fmaf(xv[i].z, wv[j].z, v);
                    v = __builtin_fmaf(xv[i].w, wv[j].w, v);
                    acc[i][j] = v;
                }
            }
        }
    }
    __syncthreads();

    // ---- logits to LDS: zs[token][e], row stride EMAX+1 (odd: no conflicts)
    float *zs = lds;
    constexpr int ZLD = EMAX + 1;
#pragma unroll
    for (int j = 0; j < TE; ++j) {
        const int e = eg * TE + j;
        if (e < E) {
            const float b = bias ? bias[e] : 0.0f;
#pragma unroll
            for (int i = 0; i < RT_TT; ++i) {
                float z = acc[i][j];
                if (bias) z = z + b;
                zs[(tg + RT_TG * i) * ZLD + e] = z;
            }
        }
    }
    __syncthreads();

    // ---- selection: wave g handles tokens [g*TB/4, (g+1)*TB/4)
    const int g = tid >> 6;
    for (int tt = g * (RT_TOK / 4); tt < (g + 1) * (RT_TOK / 4); ++tt) {
        const int64_t t = t0 + tt;
        if (t >= T) break;
        select_token(zs + tt * ZLD, t, E, k, renorm, lane, ids, wout);
    }
}

// Top-k of logits z [T][E] (any E): one wave per token.
__global__ __launch_bounds__(RT_THREADS) void route_select_kernel(const float *__restrict__ z,
                                                                  int64_t T, int E, int k,
                                                                  int renorm,
                                                                  int32_t *__restrict__ ids,
                                                                  float *__restrict__ wout) {
    const int64_t t = (int64_t)blockIdx.x * (RT_THREADS / 64) + (threadIdx.x >> 6);
    if (t >= T) return;
    select_token(z + t * E, t, E, k, renorm, threadIdx.x & 63, ids, wout);
}

// Lane-per-token router (E <= 16; and blocks of 16 experts for more experts
// and few tokens).  Lane l of a wave owns the chains of
// token l % TPW for R * G experts (the wave's 64 lanes are R sets of TPW =
// 64 / R tokens; set s takes G experts of its own): x is the lane's own
// operand, and the router element of each fma comes from a register that
// holds 16 consecutive h in each 16-lane row, broadcast by DPP (see
// route_lane_asm.h), so a stage of 64 h costs 64 G fmas plus 64 bf16
// widenings per lane and no LDS traffic per fma.  Each chain is still one
// fp32 fma per h in ascending order from +0, bias added at the end.
//
// A workgroup is NW compute waves (64 / R tokens x NW * R * G experts, all of
// E) and one producer wave.  Per stage the producer stages the x rows
// (16-byte chunk c of row r at place c ^ lane_swz(r), so the 16-byte reads
// of 8 or 16 consecutive rows fall on distinct banks) and every router row's
// 64 h into an LDS ring of NS stages by LDS-DMA, NS - 1 to NS stages ahead,
// waits for the next stage and meets the compute waves at a barrier; the
// compute waves only read LDS and run the fmas (a stage's operands are read
// during the previous stage's fmas).  Issuing the DMA from the compute waves
// themselves left it behind their VALU stream: measured on the Mixtral shape
// (16384 tokens, H = 4096, 8 experts), 41 us that way against 36 us with the
// producer wave.  The logits then go to LDS and one lane per token takes the
// top-k and the softmax weights; in the expert-block form (ZOUT) they go to
// a [T][E] buffer for route_select_kernel.  For more than 16 experts the
// chain per lane is as long as for 16 (H fmas), so up to a few thousand
// tokens this beats the register-tiled kernel, whose workgroups each run
// 5 to 20 chains per thread (E = 160, measured in the forward: 64 tokens
// 65 -> 50 us, 1024 tokens 115 -> 81, 4096 tokens 261 -> 204).
constexpr int RL_HS = 64;     // h per stage
constexpr int RL_NS_MAX = 6;  // ring stages at most (deeper rings measured no faster)

// Ring depth for stages of `stage` bytes and `per` DMA requests per stage:
// even (register sets alternate with the slots), at most 80 KiB (two
// workgroups per compute unit) and with (depth - 1) * per requests countable
// by the 6-bit vmcnt.
constexpr int lane_ring(int stage, int per) {
    int n = RL_NS_MAX;
    while (n > 2 && (n * stage > 80 * 1024 || (n - 1) * per > 63)) n -= 2;
    return n;
}

// Calls f(integral_constant<int, I>) for I = B .. N - 1.
template <int B, int N, class F>
__device__ __forceinline__ void lane_unroll(F &&f) {
    if constexpr (B < N) {
        f(std::integral_constant<int, B>{});
        lane_unroll<B + 1, N>(f);
    }
}

template <int G>
struct LaneRegs {
    u32x4 x[8];     // the lane's 64 bf16 of the stage
    floatx4 w[G];   // router rows: w[g][c] = w[e_g][h0 + 4 (lane % 16) + c]
};

// this lane's first operands, read and waited for
template <int G>
__device__ __forceinline__ void lane_read(LaneRegs<G> &r, const uint32_t (&ax)[8], uint32_t aw) {
    if constexpr (G == 2) {
        asm volatile(
            "ds_read_b128 %0, %10\n\tds_read_b128 %1, %11\n\tds_read_b128 %2, %12\n\t"
            "ds_read_b128 %3, %13\n\tds_read_b128 %4, %14\n\tds_read_b128 %5, %15\n\t"
            "ds_read_b128 %6, %16\n\tds_read_b128 %7, %17\n\t"
            "ds_read_b128 %8, %18\n\tds_read_b128 %9, %18 offset:256\n\t"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(r.x[0]), "=&v"(r.x[1]), "=&v"(r.x[2]), "=&v"(r.x[3]), "=&v"(r.x[4]),
              "=&v"(r.x[5]), "=&v"(r.x[6]), "=&v"(r.x[7]), "=&v"(r.w[0]), "=&v"(r.w[1])
            : "v"(ax[0]), "v"(ax[1]), "v"(ax[2]), "v"(ax[3]), "v"(ax[4]), "v"(ax[5]),
              "v"(ax[6]), "v"(ax[7]), "v"(aw)
            : "memory");
    } else {
        static_assert(G == 4, "two or four experts per lane");
        asm volatile(
            "ds_read_b128 %0, %12\n\tds_read_b128 %1, %13\n\tds_read_b128 %2, %14\n\t"
            "ds_read_b128 %3, %15\n\tds_read_b128 %4, %16\n\tds_read_b128 %5, %17\n\t"
            "ds_read_b128 %6, %18\n\tds_read_b128 %7, %19\n\t"
            "ds_read_b128 %8, %20\n\tds_read_b128 %9, %20 offset:256\n\t"
            "ds_read_b128 %10, %20 offset:512\n\tds_read_b128 %11, %20 offset:768\n\t"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(r.x[0]), "=&v"(r.x[1]), "=&v"(r.x[2]), "=&v"(r.x[3]), "=&v"(r.x[4]),
              "=&v"(r.x[5]), "=&v"(r.x[6]), "=&v"(r.x[7]), "=&v"(r.w[0]), "=&v"(r.w[1]),
              "=&v"(r.w[2]), "=&v"(r.w[3])
            : "v"(ax[0]), "v"(ax[1]), "v"(ax[2]), "v"(ax[3]), "v"(ax[4]), "v"(ax[5]),
              "v"(ax[6]), "v"(ax[7]), "v"(aw)
            : "memory");
    }
}

// one stage's fmas from cur, the next stage's operands (LDS byte offset OFF
// from the addresses ax / aw) read into nxt
template <int G, int OFF>
__device__ __forceinline__ void lane_stage(float (&acc)[G], const LaneRegs<G> &cur,
                                           LaneRegs<G> &nxt, const uint32_t (&ax)[8],
                                           uint32_t aw) {
    if constexpr (G == 2)
        lane_stage_g2<OFF, OFF>(acc, cur.x, cur.w, nxt.x, nxt.w, ax, aw);
    else
        lane_stage_g4<OFF, OFF>(acc, cur.x, cur.w, nxt.x, nxt.w, ax, aw);
}

// Place of a row's chunks in the x stage: 128-byte rows sit in one half of
// the 256 bytes the 64 banks span (row parity), so rows r and r + 2 share
// banks unless their places differ; r ^ (r >> 3) gives distinct places to
// any 8 consecutive rows and to the 8 rows of each parity among 16
// consecutive ones.
__device__ __forceinline__ int lane_swz(int r) { return (r ^ (r >> 3)) & 7; }

// s_waitcnt vmcnt(PER * n) for n == K, K - 1, .., 0
template <int PER, int K>
__device__ __forceinline__ void lane_wait_vm_k(int n) {
    if (n == K) {
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(K * PER) : "memory");
    } else if constexpr (K > 0) {
        lane_wait_vm_k<PER, K - 1>(n);
    }
}

// s_waitcnt vmcnt(PER * n), 0 <= n <= NS - 1; n == NS - 2 at every stage
// but the first and the last few
template <int PER, int NS>
__device__ __forceinline__ void lane_wait_vm(int n) {
    static_assert((NS - 1) * PER <= 63, "vmcnt range");
    if (__builtin_expect(n == NS - 2, 1)) {
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 2) * PER) : "memory");
        return;
    }
    lane_wait_vm_k<PER, NS - 1>(n);
}

// top-k and softmax weights of one token from its E logits, by one lane
template <int EP>
__device__ __forceinline__ void select_lane(const float *zrow, int64_t t, int E, int k,
                                            int renorm, int32_t *__restrict__ ids,
                                            float *__restrict__ wout) {
    uint64_t key[EP];
    float z[EP];
#pragma unroll
    for (int e = 0; e < EP; ++e) {
        z[e] = e < E ? zrow[e] : 0.0f;
        key[e] = e < E ? logit_key(z[e], e) : 0ull;
    }
    int sel_e[kMaxTopK];
    float sel_z[kMaxTopK];
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
        sel_e[j] = 0;
        sel_z[j] = 0.0f;
        if (j < k) {
            uint64_t best = key[0];
#pragma unroll
            for (int e = 1; e < EP; ++e) best = max_u64(best, key[e]);
            sel_e[j] = (int)(0xFFFFFFFFu - (uint32_t)best);
            sel_z[j] = key_logit(best);
#pragma unroll
            for (int e = 0; e < EP; ++e)
                if (key[e] == best) key[e] = 0ull;
        }
    }
    const double zmax = (double)sel_z[0];
    double denom = 0.0;
    if (renorm) {
#pragma unroll
        for (int j = 0; j < kMaxTopK; ++j)
            if (j < k) denom += exp((double)sel_z[j] - zmax);
    } else {
#pragma unroll
        for (int e = 0; e < EP; ++e)
            if (e < E) denom += exp((double)z[e] - zmax);
    }
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
        if (j < k) {
            ids[t * k + j] = sel_e[j];
            wout[t * k + j] = (float)(exp((double)sel_z[j] - zmax) / denom);
        }
    }
}

// select_lane's result for one token of E <= 16 logits (zrow, in LDS), by
// the whole wave: lane e holds expert e's key, so each of the k rounds is a
// wave-wide max (the same winners in the same order), and each lane takes
// one exponential (lane j: selected expert j, or lane e: expert e); the
// denominator adds the terms one by one in select_lane's order.  The same
// bits, in the time of two exponentials instead of 2k.
__device__ __forceinline__ void select_wave16(const float *zrow, int64_t t, int E, int k,
                                              int renorm, int lane, int32_t *__restrict__ ids,
                                              float *__restrict__ wout) {
    const float z = lane < E ? zrow[lane] : 0.0f;
    uint64_t key = lane < E ? logit_key(z, lane) : 0ull;
    int sel_e[kMaxTopK];
    float sel_z[kMaxTopK];
    int my_e = 0;
    float my_z = 0.0f;  // lane j < k: the j-th selected expert and logit
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
        sel_e[j] = 0;
        sel_z[j] = 0.0f;
        if (j < k) {
            const uint64_t best = wave_max_u64(key);
            sel_e[j] = (int)(0xFFFFFFFFu - (uint32_t)best);
            sel_z[j] = key_logit(best);
            if (key == best) key = 0ull;
            if (lane == j) {
                my_e = sel_e[j];
                my_z = sel_z[j];
            }
        }
    }
    const double zmax = (double)sel_z[0];
    const double ex_sel = exp((double)my_z - zmax);
    double denom = 0.0;
    if (renorm) {
        const uint64_t b = __builtin_bit_cast(uint64_t, ex_sel);
#pragma unroll
        for (int j = 0; j < kMaxTopK; ++j)
            if (j < k) denom += __builtin_bit_cast(double, readlane64(b, j));
    } else {
        const uint64_t b = __builtin_bit_cast(uint64_t, exp((double)z - zmax));
#pragma unroll
        for (int e = 0; e < 16; ++e)
            if (e < E) denom += __builtin_bit_cast(double, readlane64(b, e));
    }
    if (lane < k) {
        ids[t * k + lane] = my_e;
        wout[t * k + lane] = (float)(ex_sel / denom);
    }
}

// ZOUT: the workgroup takes experts blockIdx.y * EP .. (any E) and writes
// its logits (bias added) to zout [T][E] for a selection kernel; else one
// workgroup holds every expert (E <= EP) and selects in place.
template <int G, int R, int NW, int NS, bool ZOUT>
__global__ __launch_bounds__(64 * NW + 64) void route_lane_kernel(const bf16_t *__restrict__ x,
                                                             const float *__restrict__ wr,
                                                             const float *__restrict__ bias,
                                                             int64_t T, int H, int E, int k,
                                                             int renorm,
                                                             int32_t *__restrict__ ids,
                                                             float *__restrict__ wout,
                                                             float *__restrict__ zout) {
    constexpr int TPW = 64 / R;              // tokens per wave (and per workgroup)
    constexpr int EP = NW * R * G;           // experts per workgroup
    constexpr int XB = TPW * RL_HS * 2;      // bytes of a stage's x rows
    constexpr int WB = EP * RL_HS * 4;       // bytes of a stage's router rows
    constexpr int STAGE = XB + WB;
    constexpr int NXR = XB / 1024;           // wave-wide 16-byte DMA requests
    constexpr int NWR = WB / 1024;
    constexpr int PER = NXR + NWR;           // requests per stage (producer wave)
    static_assert(XB % 1024 == 0 && WB % 1024 == 0, "stages of whole requests");
    static_assert(NS % 2 == 0 && NS >= 2 && NS * STAGE <= 160 * 1024, "ring depth");
    static_assert(TPW * (EP + 1) * 4 <= NS * STAGE, "logits fit in the ring");
    // ring slots reached from one base address through the 16-bit offset of
    // ds_read; the slots past them use a second base
    constexpr int SPB = 65535 / STAGE + 1 < NS ? 65535 / STAGE + 1 : NS;
    static_assert(2 * SPB >= NS, "two base addresses cover the ring");
    __shared__ __attribute__((aligned(16))) char lds[NS * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool producer = wave == NW;
    const int tl = lane % TPW;                   // token of this lane
    const int eb = (wave * R + lane / TPW) * G;  // its first expert in the block
    const int64_t t0 = (int64_t)blockIdx.x * TPW;
    const int e0 = ZOUT ? (int)blockIdx.y * EP : 0;  // the block's first expert

    // the producer's DMA requests q of a stage: q < NXR: 8 x rows of 128
    // bytes (lane i: row 8 q + i / 8, 16-byte chunk (i % 8) ^ lane_swz(row)
    // into place i % 8); else 4 router rows of 256 bytes
    const char *src[PER];
    uint32_t dst[PER];
    int step_bytes[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        if (q < NXR) {
            const int r = q * 8 + (lane >> 3);
            const int c = (lane & 7) ^ lane_swz(r);
            const int64_t t = min<int64_t>(t0 + r, T - 1);
            src[q] = reinterpret_cast<const char *>(x + t * H) + c * 16;
            dst[q] = q * 1024;
            step_bytes[q] = RL_HS * 2;
        } else {
            const int qw = q - NXR;
            const int e = min(e0 + qw * 4 + (lane >> 4), E - 1);  // rows past E: unused copies
            src[q] = reinterpret_cast<const char *>(wr + (int64_t)e * H) + (lane & 15) * 16;
            dst[q] = XB + qw * 1024;
            step_bytes[q] = RL_HS * 4;
        }
    }
    auto issue = [&](int st) {  // stage st into ring slot st % NS
        char *slot = lds + (st % NS) * STAGE;
#pragma unroll
        for (int j = 0; j < PER; ++j)
            __builtin_amdgcn_global_load_lds((gbl_void_t *)(src[j] + (int64_t)st * step_bytes[j]),
                                             (lds_void_t *)(slot + dst[j]), 16, 0, 0);
    };

    // LDS byte addresses in ring slot 0 (set 0) and slot SPB (set 1): chunk c
    // of this lane's x row, and its router chunk (lane % 16) of expert eb
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void_t *)lds;
    uint32_t ax[2][8], aw[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
        for (int c = 0; c < 8; ++c)
            ax[b][c] = lds0 + b * SPB * STAGE + tl * (RL_HS * 2) + ((c ^ lane_swz(tl)) << 4);
        aw[b] = lds0 + b * SPB * STAGE + XB + eb * (RL_HS * 4) + (lane & 15) * 16;
    }

    const int nst = H / RL_HS;
    const int pre = min(NS, nst);
    float acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = 0.0f;
    if (producer) {
        // stages 0 .. NS - 1 in flight; before each barrier the next stage
        // has landed, after it the slot of the stage the compute waves have
        // just taken into registers is refilled
        for (int st = 0; st < pre; ++st) issue(st);
        lane_wait_vm<PER, NS>(pre - 1);  // stage 0
        __builtin_amdgcn_s_barrier();
        for (int st = 0; st + 1 < nst; ++st) {
            lane_wait_vm<PER, NS>(min(NS - 2, nst - 2 - st));  // stage st + 1
            __builtin_amdgcn_s_barrier();
            if (st + NS < nst) issue(st + NS);
        }
    } else {
        __builtin_amdgcn_s_barrier();  // stage 0 landed
        LaneRegs<G> regs[2];
        lane_read<G>(regs[0], ax[0], aw[0]);
        // stage st: its operands are in regs[st % 2]; at the barrier stage
        // st + 1 has landed and slot st % NS (read in step st - 1) is free
        auto step = [&](int st, auto slot_c) {
            constexpr int U = decltype(slot_c)::value;  // st % NS
            constexpr int NXT = (U + 1) % NS;           // slot read for stage st + 1
            constexpr int B = NXT >= SPB;
            if (st >= nst) return;
            if (st + 1 < nst) __builtin_amdgcn_s_barrier();
            // (after the last stage the reads of the next slot return unused data)
            lane_stage<G, (NXT - B * SPB) * STAGE>(acc, regs[U & 1], regs[(U + 1) & 1],
                                                   ax[B], aw[B]);
        };
        for (int st0 = 0; st0 < nst; st0 += NS)
            lane_unroll<0, NS>([&](auto u) { step(st0 + decltype(u)::value, u); });
    }
    if constexpr (ZOUT) {
        // (the producer's DMA has all been waited for: its last wait is vmcnt(0))
        if (producer) return;
        const int64_t t = t0 + tl;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int e = e0 + eb + g;
            if (e < E && t < T) zout[t * E + e] = bias ? acc[g] + bias[e] : acc[g];
        }
        return;
    }
    __syncthreads();  // no wave reads the ring any more; no DMA in flight

    // logits to LDS, zs[token][e] with an odd row stride
    float *zs = reinterpret_cast<float *>(lds);
    constexpr int ZLD = EP + 1;
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const int e = eb + g;
        if (e < E && !producer) zs[tl * ZLD + e] = bias ? acc[g] + bias[e] : acc[g];
    }
    __syncthreads();
    if (wave == 0 && lane < TPW) {
        const int64_t t = t0 + lane;
        if (t < T) select_lane<EP>(zs + lane * ZLD, t, E, k, renorm, ids, wout);
    }
}

template <int TE, int TT, int EG>
hipError_t launch_tt(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                     int32_t *ids, float *w, hipStream_t s) {
    constexpr int TOK = RT_THREADS / EG * TT;
    const int64_t blocks = (d.tokens + TOK - 1) / TOK;
    route_kernel<TE, TT, EG, 32><<<(unsigned)blocks, RT_THREADS, 0, s>>>(
        x, wr, bias, d.tokens, d.hidden, d.experts, d.top_k, d.renormalize, ids, w);
    return hipGetLastError();
}

template <int TE, int EG = 16>
hipError_t launch_te(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                     int32_t *ids, float *w, hipStream_t s) {
    // the most tokens per thread (fewest LDS reads per fma) that still
    // leaves enough workgroups per CU to hide latency
    constexpr int TG = RT_THREADS / EG;
    const int cus = device_cu_count();
    if (TG * 4 <= 64 && d.tokens >= (int64_t)TG * 4 * 4 * cus)
        return launch_tt<TE, (TG * 4 <= 64 ? 4 : 1), EG>(d, x, wr, bias, ids, w, s);
    if (d.tokens >= (int64_t)TG * 2 * 2 * cus) return launch_tt<TE, 2, EG>(d, x, wr, bias, ids, w, s);
    return launch_tt<TE, 1, EG>(d, x, wr, bias, ids, w, s);
}

template <int G, int R, int NW>
hipError_t launch_lane(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                       int32_t *ids, float *w, hipStream_t s) {
    constexpr int TPW = 64 / R;
    constexpr int STAGE = TPW * RL_HS * 2 + NW * R * G * RL_HS * 4;
    constexpr int PER = STAGE / 1024;
    const int64_t blocks = (d.tokens + TPW - 1) / TPW;
    route_lane_kernel<G, R, NW, lane_ring(STAGE, PER), false>
        <<<(unsigned)blocks, 64 * NW + 64, 0, s>>>(x, wr, bias, d.tokens, d.hidden, d.experts,
                                                   d.top_k, d.renormalize, ids, w, nullptr);
    return hipGetLastError();
}

// Any number of experts in blocks of NW * R * G per workgroup, logits
// through z [T][E], then the selection kernel (one wave per token).
template <int G, int R, int NW>
hipError_t launch_lane_z(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                         int32_t *ids, float *w, float *z, hipStream_t s) {
    constexpr int TPW = 64 / R, EP = NW * R * G;
    constexpr int STAGE = TPW * RL_HS * 2 + EP * RL_HS * 4;
    constexpr int PER = STAGE / 1024;
    const dim3 grid((unsigned)((d.tokens + TPW - 1) / TPW), (unsigned)((d.experts + EP - 1) / EP));
    route_lane_kernel<G, R, NW, lane_ring(STAGE, PER), true><<<grid, 64 * NW + 64, 0, s>>>(
        x, wr, bias, d.tokens, d.hidden, d.experts, d.top_k, d.renormalize, ids, w, z);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    route_select_kernel<<<(unsigned)((d.tokens + 3) / 4), RT_THREADS, 0, s>>>(
        z, d.tokens, d.experts, d.top_k, d.renormalize, ids, w);
    return hipGetLastError();
}

// Few-token router: one wave per token and block of 4 NQ experts; lane l
// runs the chain of expert e0 + l.  A chain is H dependent fmas whatever
// the mapping, so at a few tokens (a SIMD for every wave) the chain's
// latency is the router's time: a dependent fp32 fma issues every ~6
// cycles when both operands are in vector registers (measured; ~9 when one
// is a scalar just computed, ~20 per h in the lane-per-token kernel, whose
// lanes also widen x and meet a barrier every 64 h).  So the wave first
// widens its token's x row into LDS as fp32 (read back by broadcast: every
// lane the same address), the router rows stream through an LDS ring by
// LDS-DMA up to NS - 2 blocks of 64 h ahead (at decode sizes they come from
// HBM: the expert GEMMs between two forwards evict them), and each half
// block's operands are read into registers during the previous half's
// fmas.  The ring is unrolled by slot, so every read has its slot in the
// instruction's offset.  Same chains (one fp32 fma per h from +0, bias
// added at the end) and the same selection code as the other kernels, so
// the same bits.
namespace chain {

// dynamic LDS of the ring (NS * NQ KB) and the fp32 x row, at most 64 KB
constexpr size_t kMaxLds = 65536;

struct Half {  // 32 h: x (the same in every lane) and the lane's router row
    floatx4 x[8], w[8];
};

// Ring slot layout: row r (lane r's expert) at 256 r, its 16-byte chunk c
// at position c ^ (r % 16), so the 16 rows one read instruction touches
// for a given chunk fall on distinct banks.
template <int OFF>
__device__ __forceinline__ void read(Half &hv, const char *lds, const int (&woff)[16], int half,
                                     int xoff) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        hv.w[j] = *reinterpret_cast<const floatx4 *>(lds + OFF + woff[8 * half + j]);
        hv.x[j] = *reinterpret_cast<const floatx4 *>(lds + xoff + 16 * j);
    }
}

__device__ __forceinline__ float run(const Half &hv, float acc) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc = __builtin_fmaf(hv.x[j][c], hv.w[j][c], acc);
    return acc;
}

// The DPP form: lane n of each 16-lane row holds x[4n .. 4n+3] of the 64-h
// block (xq; every row reads the same 256 bytes, one read per block instead
// of sixteen), and the fma for h = 4n + c takes component c broadcast from
// lane n of its row (row_newbcast).  fma(x, w, acc) is the same operation
// whichever factor comes first, so the same bits.  Half 0 covers n = 0..7,
// half 1 n = 8..15; the s_nop covers a DPP source written by the previous
// vector instruction.
struct HalfW {  // 32 h of the lane's router row
    floatx4 w[8];
};
template <int OFF>
__device__ __forceinline__ void read_w(HalfW &hv, const char *lds, const int (&woff)[16],
                                       int half) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
        hv.w[j] = *reinterpret_cast<const floatx4 *>(lds + OFF + woff[8 * half + j]);
}
template <int HALF>
__device__ __forceinline__ float run_dpp(const floatx4 &xq, const HalfW &hv, float acc) {
    if constexpr (HALF == 0) {
        asm volatile(
        "s_nop 1\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w0] row_newbcast:0 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w1] row_newbcast:0 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w2] row_newbcast:0 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w3] row_newbcast:0 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w4] row_newbcast:1 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w5] row_newbcast:1 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w6] row_newbcast:1 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w7] row_newbcast:1 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w8] row_newbcast:2 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w9] row_newbcast:2 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w10] row_newbcast:2 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w11] row_newbcast:2 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w12] row_newbcast:3 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w13] row_newbcast:3 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w14] row_newbcast:3 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w15] row_newbcast:3 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w16] row_newbcast:4 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w17] row_newbcast:4 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w18] row_newbcast:4 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w19] row_newbcast:4 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w20] row_newbcast:5 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w21] row_newbcast:5 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w22] row_newbcast:5 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w23] row_newbcast:5 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w24] row_newbcast:6 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w25] row_newbcast:6 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w26] row_newbcast:6 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w27] row_newbcast:6 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w28] row_newbcast:7 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w29] row_newbcast:7 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w30] row_newbcast:7 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w31] row_newbcast:7 row_mask:0xf bank_mask:0xf\n\t"
        : [a] "+v"(acc)
        : [x0] "v"(xq[0]), [x1] "v"(xq[1]), [x2] "v"(xq[2]), [x3] "v"(xq[3]), [w0] "v"(hv.w[0][0]), [w1] "v"(hv.w[0][1]), [w2] "v"(hv.w[0][2]), [w3] "v"(hv.w[0][3]), [w4] "v"(hv.w[1][0]), [w5] "v"(hv.w[1][1]), [w6] "v"(hv.w[1][2]), [w7] "v"(hv.w[1][3]), [w8] "v"(hv.w[2][0]), [w9] "v"(hv.w[2][1]), [w10] "v"(hv.w[2][2]), [w11] "v"(hv.w[2][3]), [w12] "v"(hv.w[3][0]), [w13] "v"(hv.w[3][1]), [w14] "v"(hv.w[3][2]), [w15] "v"(hv.w[3][3]), [w16] "v"(hv.w[4][0]), [w17] "v"(hv.w[4][1]), [w18] "v"(hv.w[4][2]), [w19] "v"(hv.w[4][3]), [w20] "v"(hv.w[5][0]), [w21] "v"(hv.w[5][1]), [w22] "v"(hv.w[5][2]), [w23] "v"(hv.w[5][3]), [w24] "v"(hv.w[6][0]), [w25] "v"(hv.w[6][1]), [w26] "v"(hv.w[6][2]), [w27] "v"(hv.w[6][3]), [w28] "v"(hv.w[7][0]), [w29] "v"(hv.w[7][1]), [w30] "v"(hv.w[7][2]), [w31] "v"(hv.w[7][3]));
    } else {
        asm volatile(
        "s_nop 1\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w0] row_newbcast:8 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w1] row_newbcast:8 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w2] row_newbcast:8 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w3] row_newbcast:8 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w4] row_newbcast:9 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w5] row_newbcast:9 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w6] row_newbcast:9 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w7] row_newbcast:9 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w8] row_newbcast:10 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w9] row_newbcast:10 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w10] row_newbcast:10 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w11] row_newbcast:10 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w12] row_newbcast:11 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w13] row_newbcast:11 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w14] row_newbcast:11 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w15] row_newbcast:11 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w16] row_newbcast:12 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w17] row_newbcast:12 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w18] row_newbcast:12 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w19] row_newbcast:12 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w20] row_newbcast:13 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w21] row_newbcast:13 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w22] row_newbcast:13 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w23] row_newbcast:13 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w24] row_newbcast:14 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w25] row_newbcast:14 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w26] row_newbcast:14 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w27] row_newbcast:14 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x0], %[w28] row_newbcast:15 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x1], %[w29] row_newbcast:15 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x2], %[w30] row_newbcast:15 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %[a], %[x3], %[w31] row_newbcast:15 row_mask:0xf bank_mask:0xf\n\t"
        : [a] "+v"(acc)
        : [x0] "v"(xq[0]), [x1] "v"(xq[1]), [x2] "v"(xq[2]), [x3] "v"(xq[3]), [w0] "v"(hv.w[0][0]), [w1] "v"(hv.w[0][1]), [w2] "v"(hv.w[0][2]), [w3] "v"(hv.w[0][3]), [w4] "v"(hv.w[1][0]), [w5] "v"(hv.w[1][1]), [w6] "v"(hv.w[1][2]), [w7] "v"(hv.w[1][3]), [w8] "v"(hv.w[2][0]), [w9] "v"(hv.w[2][1]), [w10] "v"(hv.w[2][2]), [w11] "v"(hv.w[2][3]), [w12] "v"(hv.w[3][0]), [w13] "v"(hv.w[3][1]), [w14] "v"(hv.w[3][2]), [w15] "v"(hv.w[3][3]), [w16] "v"(hv.w[4][0]), [w17] "v"(hv.w[4][1]), [w18] "v"(hv.w[4][2]), [w19] "v"(hv.w[4][3]), [w20] "v"(hv.w[5][0]), [w21] "v"(hv.w[5][1]), [w22] "v"(hv.w[5][2]), [w23] "v"(hv.w[5][3]), [w24] "v"(hv.w[6][0]), [w25] "v"(hv.w[6][1]), [w26] "v"(hv.w[6][2]), [w27] "v"(hv.w[6][3]), [w28] "v"(hv.w[7][0]), [w29] "v"(hv.w[7][1]), [w30] "v"(hv.w[7][2]), [w31] "v"(hv.w[7][3]));
    }
    return acc;
}

}  // namespace chain

// NQ: router-row DMA requests per block (4 rows of 256 bytes each); NS ring
// slots, NS - 2 blocks of requests in flight.  ZOUT: logits (bias added) to
// zout [T][E] for route_select_kernel; else every expert is in the wave
// (E <= 4 NQ) and it selects in place.  Dynamic LDS: NS * NQ KB of ring,
// then the fp32 x row.
// (the body is a device function: the host pass of a kernel template whose
// own body calls generic lambdas over target builtins emits no launch stub)
template <int NQ, int NS, bool ZOUT>
__device__ __forceinline__ void route_chain(char *lds, const bf16_t *__restrict__ x,
                                            const float *__restrict__ wr,
                                            const float *__restrict__ bias, int64_t T, int H,
                                            int E, int k, int renorm,
                                            int32_t *__restrict__ ids, float *__restrict__ wout,
                                            float *__restrict__ zout) {
    constexpr int SLOT = NQ * 1024;  // bytes: 4 NQ rows of 64 fp32
    constexpr int RING = NS * SLOT;
    static_assert(NS >= 3 && (NS - 2) * NQ <= 63 && RING <= 65536, "ring");
    const int64_t t = blockIdx.x;
    const int lane = threadIdx.x;
    const int e0 = (int)blockIdx.y * 4 * NQ;
    const int e = e0 + lane;
    const bool live = lane < 4 * NQ && e < E;
    const int nb = H / 64;

    // DMA: request q of a block moves rows 4q .. 4q + 3 (lane l: row 4q +
    // l / 16 at position l % 16, i.e. chunk (l % 16) ^ (row % 16)); rows
    // past E repeat the last expert's.  Block b is the scalar offset.
    const __amdgpu_buffer_rsrc_t wres =
        __builtin_amdgcn_make_buffer_rsrc((void *)wr, 0, -1, 0x00020000);
    uint32_t voff[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const int r = 4 * q + lane / 16;
        const int c = (lane & 15) ^ (r & 15);
        voff[q] = (uint32_t)(((int64_t)min(e0 + r, E - 1) * H + 4 * c) * 4);
    }
    auto issue = [&](int blk, auto slot) {  // block blk (clamped) into a slot
        constexpr int S = decltype(slot)::value;
        const int sb = min(blk, nb - 1) * 256;
#pragma unroll
        for (int q = 0; q < NQ; ++q)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                wres, (lds_void_t *)(lds + S * SLOT + q * 1024), 16, voff[q], sb, 0, 0);
    };
    // x row -> LDS fp32, 8 bf16 per lane per step; the first 4096 h are
    // requested before the ring's first blocks, so both latencies overlap
    const bf16_t *xr = x + t * H;
    auto widen = [&](int i, const u32x4 &v) {
        const floatx4 lo = {bf16_lo(v[0]), bf16_hi(v[0]), bf16_lo(v[1]), bf16_hi(v[1])};
        const floatx4 hi = {bf16_lo(v[2]), bf16_hi(v[2]), bf16_lo(v[3]), bf16_hi(v[3])};
        *reinterpret_cast<floatx4 *>(lds + RING + 4 * i) = lo;
        *reinterpret_cast<floatx4 *>(lds + RING + 4 * i + 16) = hi;
    };
    u32x4 xv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int i = min(lane * 8 + 512 * j, H - 8);  // clamped: rewrites the last 8
        xv[j] = *reinterpret_cast<const u32x4 *>(xr + i);
    }
    lane_unroll<0, NS - 1>([&](auto s) { issue(decltype(s)::value, s); });
#pragma unroll
    for (int j = 0; j < 8; ++j) widen(min(lane * 8 + 512 * j, H - 8), xv[j]);
    for (int i = lane * 8 + 4096; i < H; i += 512)
        widen(i, *reinterpret_cast<const u32x4 *>(xr + i));

    // this lane's chunk offsets in a slot (idle lanes read row 4 NQ - 1)
    int woff[16];
    {
        const int r = min(lane, 4 * NQ - 1);
#pragma unroll
        for (int c = 0; c < 16; ++c) woff[c] = r * 256 + 16 * (c ^ (r & 15));
    }
    chain::HalfW h0, h1;
    floatx4 xq[2];  // the x quads of blocks of even and odd index
    const int xl = RING + 16 * (lane & 15);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 2) * NQ) : "memory");  // block 0 landed
    chain::read_w<0>(h0, lds, woff, 0);
    xq[0] = *reinterpret_cast<const floatx4 *>(lds + xl);

    float acc = 0.0f;
    int blk = 0;
    // block blk in slot S: its second half is read during the first half's
    // fmas; then block blk + 1 has landed, block blk + NS - 1 is requested
    // into the slot block blk - 1 left, and the first half of block blk + 1
    // (and its x quad) is read during the second half's fmas.  NS is even,
    // so the slot's parity is the block's.
    static_assert(NS % 2 == 0, "x quads alternate with the slot's parity");
    auto body = [&](auto slot) {
        constexpr int S = decltype(slot)::value;
        if (blk >= nb) return;
        chain::read_w<S * SLOT>(h1, lds, woff, 1);
        __builtin_amdgcn_sched_barrier(0);  // the reads go out before the fmas
        acc = chain::run_dpp<0>(xq[S & 1], h0, acc);
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 3) * NQ) : "memory");
        issue(blk + NS - 1, std::integral_constant<int, (S + NS - 1) % NS>{});
        chain::read_w<((S + 1) % NS) * SLOT>(h0, lds, woff, 0);
        xq[(S + 1) & 1] =
            *reinterpret_cast<const floatx4 *>(lds + xl + min(blk + 1, nb - 1) * 256);
        __builtin_amdgcn_sched_barrier(0);
        acc = chain::run_dpp<1>(xq[S & 1], h1, acc);
        __builtin_amdgcn_sched_barrier(0);
        ++blk;
    };
    while (blk < nb) lane_unroll<0, NS>(body);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the clamped tail requests

    const float z = bias && live ? acc + bias[e] : acc;
    if constexpr (ZOUT) {
        if (live) zout[t * E + e] = z;
        return;
    }
    float *zs = reinterpret_cast<float *>(lds);
    __syncthreads();  // every ring read done before the logits reuse it
    zs[lane] = z;
    __syncthreads();
    if (E <= 16) {
        select_wave16(zs, t, E, k, renorm, lane, ids, wout);
    } else {
        select_token(zs, t, E, k, renorm, lane, ids, wout);
    }
}

template <int NQ, int NS, bool ZOUT>
__global__ __launch_bounds__(64) void route_chain_kernel(const bf16_t *__restrict__ x,
                                                         const float *__restrict__ wr,
                                                         const float *__restrict__ bias,
                                                         int64_t T, int H, int E, int k,
                                                         int renorm, int32_t *__restrict__ ids,
                                                         float *__restrict__ wout,
                                                         float *__restrict__ zout) {
    extern __shared__ __attribute__((aligned(16))) char lds[];
    route_chain<NQ, NS, ZOUT>(lds, x, wr, bias, T, H, E, k, renorm, ids, wout, zout);
}

template <int NQ, int NS>
hipError_t launch_chain_q(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                          int32_t *ids, float *w, float *z, hipStream_t s) {
    const dim3 grid((unsigned)d.tokens, (unsigned)((d.experts + 4 * NQ - 1) / (4 * NQ)));
    const size_t lds = (size_t)NS * NQ * 1024 + (size_t)d.hidden * 4;
    if (d.experts <= 4 * NQ) {
        route_chain_kernel<NQ, NS, false><<<grid, 64, lds, s>>>(
            x, wr, bias, d.tokens, d.hidden, d.experts, d.top_k, d.renormalize, ids, w, nullptr);
        return hipGetLastError();
    }
    route_chain_kernel<NQ, NS, true><<<grid, 64, lds, s>>>(
        x, wr, bias, d.tokens, d.hidden, d.experts, d.top_k, d.renormalize, ids, w, z);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    route_select_kernel<<<(unsigned)((d.tokens + 3) / 4), RT_THREADS, 0, s>>>(
        z, d.tokens, d.experts, d.top_k, d.renormalize, ids, w);
    return hipGetLastError();
}

// up to 8 experts: one wave of 8 chains; up to 16: one of 16; more: blocks
// of 16 experts (a wave each) and the selection kernel
constexpr int kChainSlots = 8;
int chain_requests(const moe_dims &d) { return d.experts <= 8 ? 2 : 4; }
bool chain_fits(const moe_dims &d) {
    return (size_t)kChainSlots * chain_requests(d) * 1024 + (size_t)d.hidden * 4 <=
           chain::kMaxLds;
}
hipError_t launch_chain(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                        int32_t *ids, float *w, float *z, hipStream_t s) {
    if (chain_requests(d) == 2)
        return launch_chain_q<2, kChainSlots>(d, x, wr, bias, ids, w, z, s);
    return launch_chain_q<4, kChainSlots>(d, x, wr, bias, ids, w, z, s);
}

// Per-SIMD fma work of a lane-router shape: every wave issues (G + 1) VALU
// instructions per h (G fmas and one widening); waves beyond one per SIMD
// queue behind each other.
double lane_cost(int64_t tokens, int tpw, int waves_per_block, int g) {
    const double waves = (double)((tokens + tpw - 1) / tpw) * waves_per_block;
    const double simds = 4.0 * device_cu_count();
    return (waves > simds ? waves / simds : 1.0) * (g + 1);
}

// Two experts per lane (the most waves, each with the fewest instructions
// per h) up to 8 experts at every batch size measured (64 to 65536 tokens);
// 9 to 16 experts take four per lane once the batch fills every SIMD with
// two-expert waves (measured, E = 16, H = 6144: 8192 tokens 51 us with two
// against 73 us with four, 16384 tokens 85 against 76 us).
hipError_t launch_lane_router(const moe_dims &d, const bf16_t *x, const float *wr,
                              const float *bias, int32_t *ids, float *w, hipStream_t s) {
    if (d.experts <= 4) return launch_lane<2, 1, 2>(d, x, wr, bias, ids, w, s);
    if (d.experts <= 8) return launch_lane<2, 1, 4>(d, x, wr, bias, ids, w, s);
    if (lane_cost(d.tokens, 64, 4, 4) < lane_cost(d.tokens, 32, 4, 2))
        return launch_lane<4, 1, 4>(d, x, wr, bias, ids, w, s);
    return launch_lane<2, 2, 4>(d, x, wr, bias, ids, w, s);
}

}  // namespace

hipError_t launch_route(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                        int32_t *ids, float *w, float *logits, hipStream_t s) {
    if (d.tokens <= 0) return hipSuccess;
    // few tokens: the chain-per-lane kernel (its 16-byte loads of x need
    // the rows 16-byte aligned; more than 16 experts need the logits buffer;
    // measured against the lane kernels, Mixtral and DBRX shapes: faster up
    // to 256 tokens, even at 1024, slower at 4096)
    const int64_t chain_waves =
        d.tokens * ((d.experts + 4 * chain_requests(d) - 1) / (4 * chain_requests(d)));
    if (chain_waves <= kRouteChainMaxWaves && chain_fits(d) && ((uintptr_t)x & 15) == 0 &&
        (d.experts <= 16 || logits))
        return launch_chain(d, x, wr, bias, ids, w, logits, s);
    if (d.experts <= 16) return launch_lane_router(d, x, wr, bias, ids, w, s);
    // many experts, up to kRouteLogitsMaxTokens tokens: the register-tiled
    // kernel has too few workgroups to cover its serial h loop (or, up to
    // 4096 tokens, issues more instructions per chain than the lane kernel
    // does in parallel), so the lane-per-token kernel takes blocks of 16
    // experts per workgroup (logits through the caller's buffer, then the
    // selection kernel)
    if (logits && d.tokens <= kRouteLogitsMaxTokens)
        return launch_lane_z<2, 2, 4>(d, x, wr, bias, ids, w, logits, s);
    // 129..160 experts below 65536 tokens: 32 expert groups of 5, with the
    // most tokens per thread that keeps ~2 waves per SIMD (T / 4096, at most
    // 4).  Against 16 groups of 10 it reads fewer operands per fma at equal
    // occupancy, or doubles the occupancy of small batches (E = 160,
    // measured: T = 4096 279 vs 333 us, 16384 502 vs 577 us, 32768 938 vs
    // 1094 us).  From 65536 tokens 16 groups of 10 x 4 tokens is faster.
    if (d.experts > 128 && d.experts <= 160 && d.tokens < 65536) {
        if (d.tokens >= 16384) return launch_tt<5, 4, 32>(d, x, wr, bias, ids, w, s);
        if (d.tokens >= 8192) return launch_tt<5, 2, 32>(d, x, wr, bias, ids, w, s);
        return launch_tt<5, 1, 32>(d, x, wr, bias, ids, w, s);
    }
    const int te = (d.experts + 15) / 16;
    if (te <= 2) return launch_te<2>(d, x, wr, bias, ids, w, s);
    if (te <= 4) return launch_te<4>(d, x, wr, bias, ids, w, s);
    if (te <= 8) return launch_te<8>(d, x, wr, bias, ids, w, s);
    if (te <= 10) return launch_te<10>(d, x, wr, bias, ids, w, s);
    return launch_te<16>(d, x, wr, bias, ids, w, s);
}

}  // namespace moe
