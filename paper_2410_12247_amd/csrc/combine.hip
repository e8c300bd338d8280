// Combine (LocalReduce): y[t] (+)= sum_j w[t][j] * y_perm[slot_row[t*k+j]]
// for tokens t in [t_begin, t_end) over the token's slots whose local
// expert lies in [e_first, e_first + e_count), terms in ascending expert
// order, one fp32 fma each.  Adding the stages of a pipeline one after
// another therefore performs exactly the same fma sequence as a single call
// over all experts and tokens.
//
// One wave per token (and, for small batches, per range of the hidden
// dimension: blockIdx.y): the wave reads the token's k slot records, orders
// the selected ones by expert id (each ranked by counting smaller ids), then
// streams its range in 16-byte vectors, four per lane per pass; a pass
// issues the loads of all of the token's rows before its first fma, so the
// rows' loads are in flight together (KS, the most rows a token can have
// here, bounds the registers this takes).  Every output element's sum is
// the same fma sequence however the range is cut.
#include "common.h"

namespace moe {
namespace {

// y_perm rows and y are each touched once: streaming (nontemporal) access
// keeps them from evicting reusable lines from the caches
__device__ __forceinline__ float4 load_stream(const float4 *p) {
    return __builtin_bit_cast(float4,
                              __builtin_nontemporal_load(reinterpret_cast<const floatx4 *>(p)));
}
__device__ __forceinline__ void store_stream(float4 *p, float4 v) {
    __builtin_nontemporal_store(__builtin_bit_cast(floatx4, v), reinterpret_cast<floatx4 *>(p));
}

template <int KS>
__global__ __launch_bounds__(256) void combine_kernel(int64_t t_begin, int64_t t_end, int H,
                                                      int k, int e0,
                                                      int e_lo, int e_hi,
                                                      const float *__restrict__ y_perm,
                                                      const int32_t *__restrict__ ids,
                                                      const int32_t *__restrict__ slot_row,
                                                      const float *__restrict__ w,
                                                      float *__restrict__ y, int accumulate) {
    const int lane = threadIdx.x & 63;
    const int64_t t = t_begin + (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= t_end) return;
    // slot records of this token (wave-uniform after readlane)
    int my_e = 1 << 30, my_r = -1;
    float my_w = 0.f;
    if (lane < k) {
        const int e = ids[t * k + lane] - e0;
        const int r = slot_row[t * k + lane];
        if (e >= e_lo && e < e_hi && r >= 0) {
            my_e = e;
            my_r = r;
            my_w = w[t * k + lane];
        }
    }
    // uniform copies of the k records; rank each selected slot by expert id
    int se[kMaxTopK], sr[kMaxTopK];
    float sw[kMaxTopK];
    bool sv[kMaxTopK];
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
        se[j] = __builtin_amdgcn_readlane(my_e, j);
        sr[j] = __builtin_amdgcn_readlane(my_r, j);
        sw[j] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_w), j));
        sv[j] = j < k && sr[j] >= 0;
    }
    int n = 0;
    int orow[kMaxTopK];
    float ow[kMaxTopK];
#pragma unroll
    for (int p = 0; p < kMaxTopK; ++p) {
        orow[p] = 0;
        ow[p] = 0.f;
    }
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
        if (!sv[j]) continue;
        int rank = 0;
#pragma unroll
        for (int q = 0; q < kMaxTopK; ++q)
            if (sv[q] && se[q] < se[j]) ++rank;
#pragma unroll
        for (int p = 0; p < kMaxTopK; ++p)
            if (p == rank) {
                orow[p] = sr[j];
                ow[p] = sw[j];
            }
        ++n;
    }
    if (n == 0 && accumulate) return;
    const int vecs = H / 4;  // H is a multiple of 64: vecs is a multiple of 16
    // this wave's range of vectors: whole passes of 256
    const int np = (vecs + 255) / 256;
    const int per = (np + (int)gridDim.y - 1) / (int)gridDim.y * 256;
    const int v_lo = (int)blockIdx.y * per, v_hi = min(vecs, v_lo + per);
    float4 *yrow = reinterpret_cast<float4 *>(y + t * H);
    // four 16-byte vectors per lane per pass: all loads of a pass in flight
    for (int v0 = v_lo + lane; v0 < v_hi; v0 += 256) {
        float4 acc[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int v = min(v0 + 64 * u, vecs - 1);
            acc[u] = accumulate ? load_stream(yrow + v) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        // every row's loads first, then the fmas in ascending expert order
        float4 p[KS][4];
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            if (j < n) {
                const float4 *prow =
                    reinterpret_cast<const float4 *>(y_perm + (int64_t)orow[j] * H);
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    p[j][u] = load_stream(prow + min(v0 + 64 * u, vecs - 1));
            }
        }
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            if (j < n) {
                const float c = ow[j];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    acc[u].x = __builtin_fmaf(c, p[j][u].x, acc[u].x);
                    acc[u].y = __builtin_fmaf(c, p[j][u].y, acc[u].y);
                    acc[u].z = __builtin_fmaf(c, p[j][u].z, acc[u].z);
                    acc[u].w = __builtin_fmaf(c, p[j][u].w, acc[u].w);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (v0 + 64 * u < v_hi) store_stream(yrow + v0 + 64 * u, acc[u]);
    }
}

}  // namespace

hipError_t launch_combine(const moe_dims &d, int e_first, int e_count, int64_t t_begin,
                          int64_t t_end, const float *y_perm, const int32_t *ids,
                          const int32_t *slot_row, const float *w, float *y, int accumulate,
                          hipStream_t s) {
    if (t_end <= t_begin) return hipSuccess;
    const int64_t blocks = (t_end - t_begin + 3) / 4;
    // few tokens: each token's passes over the hidden dimension spread over
    // workgroups of their own, so they run side by side instead of one
    // after another (a pass waits for its rows' loads)
    const int passes = (d.hidden / 4 + 255) / 256;
    const int split = blocks * passes <= 2 * (int64_t)device_cu_count() * 4 ? passes : 1;
    // a token has at most k rows in range
    const int ks = d.top_k;
    auto go = [&](auto kernel) {
        kernel<<<dim3((unsigned)blocks, (unsigned)split), 256, 0, s>>>(
            t_begin, t_end, d.hidden, d.top_k, d.local_begin, e_first, e_first + e_count, y_perm,
            ids, slot_row, w, y, accumulate);
        return hipGetLastError();
    };
    if (ks <= 1) return go(combine_kernel<1>);
    if (ks <= 2) return go(combine_kernel<2>);
    if (ks <= 4) return go(combine_kernel<4>);
    return go(combine_kernel<kMaxTopK>);
}

}  // namespace moe
