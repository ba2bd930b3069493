// Data movement of the channel saliency (FlexMoE Sec. 3.1, Eq. 2) around
// its backward GEMMs (gemm_bwd.hip):
//   - transposed weight copies (W_down^T [E][I][d] is the B operand of the
//     dgrad and the theta of the down matrix's saliency; the training
//     backward also takes W_gate^T and W_up^T);
//   - transposed copies of x and of dO = w_a dY_t for the routed rows, whose
//     segments become the reduction dimension of the wgrad, and dO itself;
//   - the final sum of the wgrad tiles' partial scores.
// Transposes go through a 64 x 64 LDS tile with 16-byte global accesses on
// both sides.
#include "saliency.h"
#include "train.h"

namespace flexmoe {

namespace {
constexpr int TT = 64;        // transpose tile
constexpr int TPAD = TT + 2;  // LDS row pitch (bf16): odd word stride spreads the column reads
constexpr int TTHREADS = 256;

__device__ __forceinline__ void put8(bf16_t* dst, uint4 v) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        dst[2 * i] = (bf16_t)(w[i] & 0xffffu);
        dst[2 * i + 1] = (bf16_t)(w[i] >> 16);
    }
}

__device__ __forceinline__ uint4 pack8(const bf16_t* v) {
    return make_uint4((uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16),
                      (uint32_t)v[4] | ((uint32_t)v[5] << 16), (uint32_t)v[6] | ((uint32_t)v[7] << 16));
}
}  // namespace

// src [batch][R][C] -> dst [batch][C][R] (e.g. W_down [E][d][I] -> W_down^T
// [E][I][d]); block (column tile, row tile, batch).  The names below follow
// that example: rows n < d, columns c < I.
__global__ __launch_bounds__(TTHREADS) void transpose_batched_kernel(const bf16_t* __restrict__ wd,
                                                                     bf16_t* __restrict__ wdt, int d, int I) {
    __shared__ bf16_t tile[TT][TPAD];
    const size_t e = blockIdx.z;
    const int c0 = blockIdx.x * TT, n0 = blockIdx.y * TT;
    const bf16_t* src = wd + e * d * I;
    bf16_t* dst = wdt + e * I * d;
    for (int k = threadIdx.x; k < TT * TT / 8; k += TTHREADS) {
        const int r = k >> 3, ch = (k & 7) * 8;  // unit row r, channels ch .. ch+7
        const int n = n0 + r, c = c0 + ch;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (n < d && c < I) v = *reinterpret_cast<const uint4*>(src + (size_t)n * I + c);
        put8(&tile[r][ch], v);
    }
    __syncthreads();
    for (int k = threadIdx.x; k < TT * TT / 8; k += TTHREADS) {
        const int r = k >> 3, ch = (k & 7) * 8;  // channel row r, units ch .. ch+7
        const int c = c0 + r, n = n0 + ch;
        if (c >= I || n >= d) continue;
        bf16_t v[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) v[t] = tile[ch + t][r];
        *reinterpret_cast<uint4*>(dst + (size_t)c * d + n) = pack8(v);
    }
}

// Padded rows q0 .. q0+63 (every routed segment takes packed_width(rows)
// rows from its prow0) x columns n0 .. n0+63 of x (blockIdx.z = 0) or of
// dO = w_a dY_t (blockIdx.z = 1), written transposed; padding rows are zeros.
__global__ __launch_bounds__(TTHREADS) void sal_prep_kernel(SalPrepParams p) {
    __shared__ bf16_t tile[TT][TPAD];
    const SegMeta last = p.seg[p.nseg - 1];
    const int ptot = last.e >= 0 ? last.prow0 + packed_width(last.rows) : 0;
    const int q0 = blockIdx.x * TT, n0 = blockIdx.y * TT;
    if (q0 >= ptot) return;
    const bool grad = blockIdx.z == 1;
    for (int k = threadIdx.x; k < TT * TT / 8; k += TTHREADS) {
        const int r = k >> 3, ch = (k & 7) * 8;
        const int q = q0 + r, n = n0 + ch;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (q < ptot && n < p.d) {
            // routed segment of padded row q: the last one starting at or before q
            int lo = p.hs, hi = p.nseg - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (p.seg[mid].prow0 <= q) lo = mid;
                else hi = mid - 1;
            }
            const SegMeta sm = p.seg[lo];
            const int loc = q - sm.prow0;
            if (loc < sm.rows) {
                const int row = sm.row0 + loc;
                const int a = p.perm[row];
                const size_t src = (size_t)(a / p.k) * p.d + n;
                if (!grad) {
                    v = *reinterpret_cast<const uint4*>(p.x + src);
                } else {
                    const float w = p.wts[a];
                    const float4 f0 = *reinterpret_cast<const float4*>(p.dy + src);
                    const float4 f1 = *reinterpret_cast<const float4*>(p.dy + src + 4);
                    const bf16_t b[8] = {f32_to_bf16(w * f0.x), f32_to_bf16(w * f0.y), f32_to_bf16(w * f0.z),
                                         f32_to_bf16(w * f0.w), f32_to_bf16(w * f1.x), f32_to_bf16(w * f1.y),
                                         f32_to_bf16(w * f1.z), f32_to_bf16(w * f1.w)};
                    v = pack8(b);
                    *reinterpret_cast<uint4*>(p.dO + (size_t)row * p.d + n) = v;
                }
            }
        }
        put8(&tile[r][ch], v);
    }
    __syncthreads();
    bf16_t* out = grad ? p.dot : p.xt;
    for (int k = threadIdx.x; k < TT * TT / 8; k += TTHREADS) {
        const int r = k >> 3, ch = (k & 7) * 8;  // column n0 + r, padded rows q0+ch .. +7
        const int n = n0 + r, q = q0 + ch;
        if (n >= p.d || q >= ptot) continue;  // ptot and q are multiples of 8
        bf16_t v[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) v[t] = tile[ch + t][r];
        *reinterpret_cast<uint4*>(out + (size_t)n * p.ldt + q) = pack8(v);
    }
}

// scores[e][c] += scale * (sum over the three matrices and their partial
// sums, in that fixed order).
__global__ __launch_bounds__(256) void sal_reduce_kernel(const float* __restrict__ partial, int EI, int parts,
                                                         float scale, float* __restrict__ scores) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= EI) return;
    float s = 0.f;
    for (int m = 0; m < 3; ++m) {
        const float* pp = partial + ((size_t)m * EI + i) * parts;
        for (int q = 0; q < parts; ++q) s += pp[q];
    }
    scores[i] += scale * s;
}

hipError_t launch_transpose_batched(const bf16_t* src, bf16_t* dst, int batch, int rows, int cols,
                                    hipStream_t s) {
    if (batch <= 0 || rows <= 0 || cols <= 0) return hipSuccess;
    const dim3 grid(ceil_div(cols, TT), ceil_div(rows, TT), batch);
    transpose_batched_kernel<<<grid, TTHREADS, 0, s>>>(src, dst, rows, cols);
    return hipGetLastError();
}

hipError_t launch_sal_prep(const SalPrepParams& p, hipStream_t s) {
    const dim3 grid(ceil_div(p.ldt, TT), ceil_div(p.d, TT), 2);
    sal_prep_kernel<<<grid, TTHREADS, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_sal_reduce(const float* partial, int E, int I, int parts, float scale, float* scores,
                             hipStream_t s) {
    const int EI = E * I;
    sal_reduce_kernel<<<ceil_div(EI, 256), 256, 0, s>>>(partial, EI, parts, scale, scores);
    return hipGetLastError();
}

}  // namespace flexmoe
