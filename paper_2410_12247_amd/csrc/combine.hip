// Combine (LocalReduce): y[t] (+)= sum_j w[t][j] * y_perm[slot_row[t*k+j]]
// for tokens t in [t_begin, t_end) over the token's slots whose local
// expert lies in [e_first, e_first + e_count), terms in ascending expert
// order, one fp32 fma each.  Adding the stages of a pipeline one after
// another therefore performs exactly the same fma sequence as a single call
// over all experts and tokens.
//
// One wave per token: the wave reads the token's k slot records, orders the
// selected ones by expert id (each ranked by counting smaller ids), then streams
// the hidden dimension in 16-byte vectors.
#include "common.h"

namespace moe {
namespace {

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
    const int vecs = H / 4;
    float4 *yrow = reinterpret_cast<float4 *>(y + t * H);
    for (int v = lane; v < vecs; v += 64) {
        float4 acc = accumulate ? yrow[v] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int j = 0; j < kMaxTopK; ++j) {
            if (j < n) {
                const float4 p =
                    reinterpret_cast<const float4 *>(y_perm + (int64_t)orow[j] * H)[v];
                const float c = ow[j];
                acc.x = __builtin_fmaf(c, p.x, acc.x);
                acc.y = __builtin_fmaf(c, p.y, acc.y);
                acc.z = __builtin_fmaf(c, p.z, acc.z);
                acc.w = __builtin_fmaf(c, p.w, acc.w);
            }
        }
        yrow[v] = acc;
    }
}

}  // namespace

hipError_t launch_combine(const moe_dims &d, int e_first, int e_count, int64_t t_begin,
                          int64_t t_end, const float *y_perm, const int32_t *ids,
                          const int32_t *slot_row, const float *w, float *y, int accumulate,
                          hipStream_t s) {
    if (t_end <= t_begin) return hipSuccess;
    const int64_t blocks = (t_end - t_begin + 3) / 4;
    combine_kernel<<<(unsigned)blocks, 256, 0, s>>>(t_begin, t_end, d.hidden, d.top_k,
                                                    d.local_begin, e_first, e_first + e_count,
                                                    y_perm, ids, slot_row, w, y, accumulate);
    return hipGetLastError();
}

}  // namespace moe
