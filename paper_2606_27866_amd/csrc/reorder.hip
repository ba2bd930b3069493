// One-time channel ranking and reorder (FlexMoE Sec. 3.1, Eq. 3).
//   rank_kernel: position of channel c in the stable descending order of the
//     scores = #{j : (s_j, j) precedes (s_c, c)}, with NaN after every
//     number.  The order is total, so the positions form a permutation and
//     perm[e][position] = c.
//   gather_rows_kernel: W~_gate[e][c] = W_gate[e][perm[e][c]] (and up).
//   gather_cols_kernel: W~_down[e][n][c] = W_down[e][n][perm[e][c]].
#include "kernels.h"

namespace flexmoe {

__device__ __forceinline__ bool score_before(float va, int ia, float vb, int ib) {
    const bool na = __builtin_isnan(va), nb = __builtin_isnan(vb);
    if (na != nb) return nb;
    if (!na && va != vb) return va > vb;
    return ia < ib;
}

__global__ __launch_bounds__(256) void rank_kernel(const float* __restrict__ scores, int I,
                                                   int32_t* __restrict__ perm) {
    constexpr int CH = 2048;
    __shared__ float sc[CH];
    const int e = blockIdx.y;
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    const float* s = scores + (size_t)e * I;
    const float vc = c < I ? s[c] : 0.f;
    int rank = 0;
    for (int j0 = 0; j0 < I; j0 += CH) {
        const int n = min(CH, I - j0);
        __syncthreads();
        for (int j = threadIdx.x; j < n; j += blockDim.x) sc[j] = s[j0 + j];
        __syncthreads();
        if (c < I)
            for (int j = 0; j < n; ++j) rank += score_before(sc[j], j0 + j, vc, c) ? 1 : 0;
    }
    if (c < I) perm[(size_t)e * I + rank] = c;
}

// one block per (expert, ranked channel); rows are copied in 16-byte pieces
__global__ __launch_bounds__(128) void gather_rows_kernel(const uint8_t* __restrict__ wg,
                                                          const uint8_t* __restrict__ wu,
                                                          uint8_t* __restrict__ wg_r,
                                                          uint8_t* __restrict__ wu_r,
                                                          const int32_t* __restrict__ perm, int I,
                                                          size_t row_bytes) {
    const size_t e = blockIdx.y, c = blockIdx.x;
    const size_t src = (e * I + (size_t)perm[e * I + c]) * row_bytes;
    const size_t dst = (e * I + c) * row_bytes;
    for (size_t b = threadIdx.x * 16; b < row_bytes; b += blockDim.x * 16) {
        *reinterpret_cast<u32x4*>(wg_r + dst + b) = *reinterpret_cast<const u32x4*>(wg + src + b);
        *reinterpret_cast<u32x4*>(wu_r + dst + b) = *reinterpret_cast<const u32x4*>(wu + src + b);
    }
}

template <typename T>
__global__ __launch_bounds__(256) void gather_cols_kernel(const T* __restrict__ wd, T* __restrict__ wd_r,
                                                          const int32_t* __restrict__ perm, int I, int d) {
    const size_t e = blockIdx.y, n = blockIdx.x;
    const T* src = wd + (e * d + n) * (size_t)I;
    T* dst = wd_r + (e * d + n) * (size_t)I;
    const int32_t* pe = perm + e * I;
    for (int c = threadIdx.x; c < I; c += blockDim.x) dst[c] = src[pe[c]];
}

hipError_t launch_rank_reorder(const float* scores, const void* wg, const void* wu, const void* wd,
                               void* wg_r, void* wu_r, void* wd_r, int32_t* perm, int E, int I,
                               int d, int esize, hipStream_t s) {
    rank_kernel<<<dim3(ceil_div(I, 256), E), 256, 0, s>>>(scores, I, perm);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    gather_rows_kernel<<<dim3(I, E), 128, 0, s>>>((const uint8_t*)wg, (const uint8_t*)wu,
                                                   (uint8_t*)wg_r, (uint8_t*)wu_r, perm, I,
                                                   (size_t)d * esize);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    if (esize == 2)
        gather_cols_kernel<bf16_t><<<dim3(d, E), 256, 0, s>>>((const bf16_t*)wd, (bf16_t*)wd_r, perm, I, d);
    else
        gather_cols_kernel<float><<<dim3(d, E), 256, 0, s>>>((const float*)wd, (float*)wd_r, perm, I, d);
    return hipGetLastError();
}

}  // namespace flexmoe
