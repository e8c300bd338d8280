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

// Logits phase layout: 256 threads = TG token groups x EG expert groups
// (EG = 16, or 8 when E <= 8 so that no thread repeats an expert); a thread
// owns TT tokens (tg + TG i: consecutive lanes read rows 36 floats apart, so
// eight lanes of a 16-byte LDS read land on distinct banks) x TE experts
// (TE = ceil(E / EG)) and keeps their fma chains in registers.  x and the
// router are staged through two LDS buffers HC h at a time: the router rows
// by LDS-DMA, x through registers (widened to fp32), the next chunk in
// flight while the current one is multiplied; per 4 h a thread reads
// TT + TE float4 and issues 4*TT*TE fmas.  With few experts the fmas per
// chunk are few, so the chunk is longer (HC = 128) to keep more bytes in
// flight per wait.
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

// Half a stage's operands of the streaming router, read together with one
// wait: this thread's four 16-byte x chunks and its expert's 32 router
// weights (eight 16-byte reads from one base).  Written out because the
// compiler puts a full vmcnt(0) in front of LDS reads that may alias the
// LDS-DMA requests in flight, which drains the ring every stage; the ring's
// own vmcnt wait and barrier order the data (the slot read here landed for
// every wave before the barrier, and is refilled only after the next one).
__device__ __forceinline__ void stream_half_operands(u32x4 (&v)[4], floatx4 (&w)[8],
                                                     const uint32_t (&a)[4], uint32_t wa) {
    asm volatile(
        "ds_read_b128 %0, %12\n\t"
        "ds_read_b128 %1, %13\n\t"
        "ds_read_b128 %2, %14\n\t"
        "ds_read_b128 %3, %15\n\t"
        "ds_read_b128 %4, %16\n\t"
        "ds_read_b128 %5, %16 offset:16\n\t"
        "ds_read_b128 %6, %16 offset:32\n\t"
        "ds_read_b128 %7, %16 offset:48\n\t"
        "ds_read_b128 %8, %16 offset:64\n\t"
        "ds_read_b128 %9, %16 offset:80\n\t"
        "ds_read_b128 %10, %16 offset:96\n\t"
        "ds_read_b128 %11, %16 offset:112\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(w[0]), "=&v"(w[1]),
          "=&v"(w[2]), "=&v"(w[3]), "=&v"(w[4]), "=&v"(w[5]), "=&v"(w[6]), "=&v"(w[7])
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(wa)
        : "memory");
}

// Streaming router: workgroup = TB tokens x EB experts (TB * EB = 256), one
// fma chain per thread.  x rows (bf16) and router rows (fp32) stream through
// an LDS ring of RS_NS stages of RS_HS h by LDS-DMA, RS_NS - 1 stages in
// flight, so the latency of the loads is covered even when each stage holds
// little work (few tokens, or few experts).  Each wave issues the same
// number of DMA requests per stage (short waves repeat their last request:
// the same bytes to the same place), so one vmcnt wait per stage is right
// for every wave.  x chunks are XOR-swizzled by row so the 16 rows a wave
// reads at once spread over the banks.
// The logits go to z [T][E] and route_select_kernel picks.  (A fused form
// for E <= 16, the workgroup picking the top-k of its tokens itself, was
// slower than route_kernel at every T.)
constexpr int RS_HS = 64;  // h per stage (two halves of four 16-byte x chunks)
constexpr int RS_NS = 8;   // stages in the ring
template <int TB, int EB>
__global__ __launch_bounds__(RT_THREADS) void route_stream_kernel(
    const bf16_t *__restrict__ x, const float *__restrict__ wr, const float *__restrict__ bias,
    int64_t T, int H, int E, float *__restrict__ z) {
    static_assert(TB * EB == RT_THREADS, "one chain per thread");
    static_assert(RS_HS == 64, "stage reads: 8 x chunks of 8 h, 2 x 32 weights");
    constexpr int XB = TB * RS_HS * 2;    // bytes of an x stage
    constexpr int WB = EB * RS_HS * 4;    // bytes of a router stage
    constexpr int NXI = XB / 1024;        // wave-wide 16-byte DMA requests
    constexpr int NWI = WB / 1024;
    constexpr int PER = (NXI + NWI + 3) / 4;  // requests per wave per stage
    static_assert(XB % 1024 == 0 && WB % 1024 == 0, "stages of whole requests");
    static_assert((RS_NS - 2) * PER <= 63, "vmcnt range");
    constexpr int STAGE = XB + WB;
    __shared__ __attribute__((aligned(16))) char lds[RS_NS * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tb = tid % TB;   // token of this thread's chain
    const int eb = tid / TB;   // expert
    const int64_t t0 = (int64_t)blockIdx.x * TB;
    const int e0 = blockIdx.y * EB;

    // this wave's requests: q = wave + 4 j (j < PER), clamped to the last
    // real one; q < NXI are x requests (8 rows of 128 bytes), the rest
    // router requests (4 rows of 256 bytes)
    const char *src[PER];
    int dst[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int q = min(wave + 4 * j, NXI + NWI - 1);
        if (q < NXI) {
            const int r = q * 8 + (lane >> 3);
            const int c = (lane & 7) ^ (r & 7);  // 16-byte chunk of the row this lane fetches
            const int64_t t = min<int64_t>(t0 + r, T - 1);
            src[j] = reinterpret_cast<const char *>(x + t * H) + c * 16;
            dst[j] = q * 1024;
        } else {
            const int qw = q - NXI;
            const int r = qw * 4 + (lane >> 4);
            const int e = min(e0 + r, E - 1);  // rows past E: a copy, never used
            src[j] = reinterpret_cast<const char *>(wr + (int64_t)e * H) + (lane & 15) * 16;
            dst[j] = XB + qw * 1024;
        }
    }
    auto issue = [&](int st) {  // stage st into ring slot st % RS_NS
        const int hb = st * RS_HS;
        char *slot = lds + (st % RS_NS) * STAGE;
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int q = min(wave + 4 * j, NXI + NWI - 1);
            const int scale = q < NXI ? 2 : 4;  // bytes per element
            __builtin_amdgcn_global_load_lds((gbl_void_t *)(src[j] + (int64_t)hb * scale),
                                             (lds_void_t *)(slot + dst[j]), 16, 0, 0);
        }
    };

    const int nst = H / RS_HS;
#pragma unroll
    for (int st = 0; st < RS_NS - 1; ++st)
        if (st < nst) issue(st);
    // LDS byte addresses in ring slot 0: chunk c of this thread's x row
    // (stored at c ^ (row % 8)), and its expert's router row
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void_t *)lds;
    uint32_t xaddr[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) xaddr[c] = lds0 + tb * (RS_HS * 2) + ((c ^ (tb & 7)) * 16);
    const uint32_t waddr = lds0 + XB + eb * (RS_HS * 4);
    float acc = 0.0f;
    for (int st = 0; st < nst; ++st) {
        // stage st landed (this wave's share; later stages may be in flight)
        if (st + RS_NS - 2 < nst) {
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"((RS_NS - 2) * PER) : "memory");
        } else {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
        // every wave's share landed; slot (st - 1) fully read (a plain
        // barrier: the waits above are the only memory ordering needed, and
        // a fenced barrier would drain the requests still in flight)
        __builtin_amdgcn_s_barrier();
        if (st + RS_NS - 1 < nst) issue(st + RS_NS - 1);
        const uint32_t sbase = (uint32_t)((st % RS_NS) * STAGE);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            uint32_t a[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = xaddr[half * 4 + i] + sbase;
            u32x4 xs[4];
            floatx4 ws[8];
            stream_half_operands(xs, ws, a, waddr + sbase + half * 128);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const u32x4 xv = xs[i];
                const floatx4 w0 = ws[2 * i], w1 = ws[2 * i + 1];
                acc = __builtin_fmaf(bf16_lo(xv.x), w0.x, acc);
                acc = __builtin_fmaf(bf16_hi(xv.x), w0.y, acc);
                acc = __builtin_fmaf(bf16_lo(xv.y), w0.z, acc);
                acc = __builtin_fmaf(bf16_hi(xv.y), w0.w, acc);
                acc = __builtin_fmaf(bf16_lo(xv.z), w1.x, acc);
                acc = __builtin_fmaf(bf16_hi(xv.z), w1.y, acc);
                acc = __builtin_fmaf(bf16_lo(xv.w), w1.z, acc);
                acc = __builtin_fmaf(bf16_hi(xv.w), w1.w, acc);
            }
        }
    }
    const int e = e0 + eb;
    const int64_t t = t0 + tb;
    if (e < E && bias) acc = acc + bias[e];
    if (e < E && t < T) z[t * E + e] = acc;
}

// Top-k of logits z [T][E] from route_stream_kernel: one wave per token.
__global__ __launch_bounds__(RT_THREADS) void route_select_kernel(const float *__restrict__ z,
                                                                  int64_t T, int E, int k,
                                                                  int renorm,
                                                                  int32_t *__restrict__ ids,
                                                                  float *__restrict__ wout) {
    const int64_t t = (int64_t)blockIdx.x * (RT_THREADS / 64) + (threadIdx.x >> 6);
    if (t >= T) return;
    select_token(z + t * E, t, E, k, renorm, threadIdx.x & 63, ids, wout);
}

template <int TE, int TT, int EG>
hipError_t launch_tt(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                     int32_t *ids, float *w, hipStream_t s) {
    constexpr int TOK = RT_THREADS / EG * TT;
    const int64_t blocks = (d.tokens + TOK - 1) / TOK;
    // longer chunks when few experts give little work per chunk (H is a
    // multiple of 64; 128-h chunks need a multiple of 128).  256-h chunks
    // wait half as often; they are taken when two workgroups still fit a
    // CU's 160 KiB of LDS, or when the grid does not fill the chip anyway
    // (measured: DBRX T = 8192 0.117 -> 0.105 ms, Mixtral T = 64 0.062 ->
    // 0.053 ms; at Mixtral T = 16384 one workgroup per CU, 0.095 -> 0.131 ms)
    if constexpr (TE == 1) {
        constexpr size_t lds256 = (2 * (size_t)TOK * (256 + 4) + 2 * (size_t)EG * 256) * 4;
        constexpr bool fits = lds256 <= 160 * 1024;
        constexpr bool two_fit = 2 * lds256 <= 160 * 1024;
        if constexpr (fits) {
            if (d.hidden % 256 == 0 && (two_fit || blocks <= device_cu_count())) {
                route_kernel<TE, TT, EG, 256><<<(unsigned)blocks, RT_THREADS, 0, s>>>(
                    x, wr, bias, d.tokens, d.hidden, d.experts, d.top_k, d.renormalize, ids, w);
                return hipGetLastError();
            }
        }
        if (d.hidden % 128 == 0)
            route_kernel<TE, TT, EG, 128><<<(unsigned)blocks, RT_THREADS, 0, s>>>(
                x, wr, bias, d.tokens, d.hidden, d.experts, d.top_k, d.renormalize, ids, w);
        else
            route_kernel<TE, TT, EG, 64><<<(unsigned)blocks, RT_THREADS, 0, s>>>(
                x, wr, bias, d.tokens, d.hidden, d.experts, d.top_k, d.renormalize, ids, w);
    } else {
        route_kernel<TE, TT, EG, 32><<<(unsigned)blocks, RT_THREADS, 0, s>>>(
            x, wr, bias, d.tokens, d.hidden, d.experts, d.top_k, d.renormalize, ids, w);
    }
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

}  // namespace

template <int EB>
hipError_t launch_stream(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                         int32_t *ids, float *w, float *z, hipStream_t s) {
    constexpr int TB = RT_THREADS / EB;
    const dim3 grid((unsigned)((d.tokens + TB - 1) / TB), (unsigned)((d.experts + EB - 1) / EB));
    route_stream_kernel<TB, EB><<<grid, RT_THREADS, 0, s>>>(x, wr, bias, d.tokens, d.hidden,
                                                            d.experts, z);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    route_select_kernel<<<(unsigned)((d.tokens + 3) / 4), RT_THREADS, 0, s>>>(
        z, d.tokens, d.experts, d.top_k, d.renormalize, ids, w);
    return hipGetLastError();
}

hipError_t launch_route(const moe_dims &d, const bf16_t *x, const float *wr, const float *bias,
                        int32_t *ids, float *w, float *logits, hipStream_t s) {
    if (d.tokens <= 0) return hipSuccess;
    if (d.experts <= 8) return launch_te<1, 8>(d, x, wr, bias, ids, w, s);
    // many experts, few tokens: the register-tiled kernel has too few
    // workgroups to cover its serial h loop, so the streaming kernel spreads
    // expert blocks over more workgroups (logits through the caller's
    // buffer, then the selection kernel).  With E <= 16 the register-tiled
    // kernel is faster at every T measured (1 to 16384 tokens).
    if (d.experts > 16 && logits && d.tokens <= kRouteStreamMaxTokens)
        return launch_stream<16>(d, x, wr, bias, ids, w, logits, s);
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
    if (te <= 1) return launch_te<1>(d, x, wr, bias, ids, w, s);
    if (te <= 2) return launch_te<2>(d, x, wr, bias, ids, w, s);
    if (te <= 4) return launch_te<4>(d, x, wr, bias, ids, w, s);
    if (te <= 8) return launch_te<8>(d, x, wr, bias, ids, w, s);
    if (te <= 10) return launch_te<10>(d, x, wr, bias, ids, w, s);
    return launch_te<16>(d, x, wr, bias, ids, w, s);
}

}  // namespace moe
