// fp32 instantiation of the two ragged grouped GEMMs (same segment and tile
// tables as the bf16 path).  Plain LDS-tiled FMA on the vector ALUs: 64 x 64
// tiles, 4 x 4 outputs per thread.  This mode exists for fp32 parity with the
// oracle on small layers; the bf16 MFMA kernels are the fast path.
#include "kernels.h"

namespace flexmoe {

namespace {
constexpr int BM = kF32BM, BN = kF32BN, BK = 16;
}

__global__ __launch_bounds__(256) void gemm1_f32_kernel(Gemm1Params<float> p) {
    __shared__ float As[BK][BM + 4];
    __shared__ float Bg[BK][BN + 4];
    __shared__ float Bu[BK][BN + 4];
    int s, local;
    SegMeta sm;
    if (!tile_of(p, blockIdx.x, s, sm, local)) return;
    const int mt = ceil_div(sm.rows, BM);
    const int mtile = local % mt, ntile = local / mt;
    const bool shared = sm.e < 0;
    const size_t wofs = shared ? 0 : routed_weights(p, sm).base;
    const float* Wg = (shared ? p.sg : p.wg) + wofs;
    const float* Wu = (shared ? p.su : p.wu) + wofs;

    const int tid = threadIdx.x;
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    const int row = mtile * BM + lr;
    const float* asrc = nullptr;
    if (row < sm.rows) {
        const int t = shared ? row : (int)min((unsigned)(p.perm[sm.row0 + row] / p.top_k), (unsigned)(p.tokens - 1));
        asrc = p.x + (size_t)t * p.d;
    }
    const int ch = ntile * BN + lr;
    const float* gsrc = ch < sm.kg ? Wg + (size_t)ch * p.d : nullptr;  // channels the GEMM computes
    const float* usrc = ch < sm.kg ? Wu + (size_t)ch * p.d : nullptr;

    const int ty = tid >> 4, tx = tid & 15;
    float ag[4][4] = {}, au[4][4] = {};
    const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int k0 = 0; k0 < p.d; k0 += BK) {
        const bool kin = k0 + lk < p.d;
        const float4 a = (asrc && kin) ? *reinterpret_cast<const float4*>(asrc + k0 + lk) : z4;
        const float4 g = (gsrc && kin) ? *reinterpret_cast<const float4*>(gsrc + k0 + lk) : z4;
        const float4 u = (usrc && kin) ? *reinterpret_cast<const float4*>(usrc + k0 + lk) : z4;
        As[lk + 0][lr] = a.x; As[lk + 1][lr] = a.y; As[lk + 2][lr] = a.z; As[lk + 3][lr] = a.w;
        Bg[lk + 0][lr] = g.x; Bg[lk + 1][lr] = g.y; Bg[lk + 2][lr] = g.z; Bg[lk + 3][lr] = g.w;
        Bu[lk + 0][lr] = u.x; Bu[lk + 1][lr] = u.y; Bu[lk + 2][lr] = u.z; Bu[lk + 3][lr] = u.w;
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < BK; ++kk) {
            float av[4], gv[4], uv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                gv[j] = Bg[kk][tx * 4 + j];
                uv[j] = Bu[kk][tx * 4 + j];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    ag[i][j] = fmaf(av[i], gv[j], ag[i][j]);
                    au[i][j] = fmaf(av[i], uv[j], au[i][j]);
                }
        }
        __syncthreads();
    }
    float* Hb = shared ? p.Hs : p.H + (size_t)sm.row0 * p.I;
    const int ldh = shared ? p.Is : p.I;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = mtile * BM + ty * 4 + i;
            const int c = ntile * BN + tx * 4 + j;
            if (r < sm.rows && c < sm.kg) {  // channels [kk, kg) are written as zeros
                const float g = ag[i][j];
                Hb[(size_t)r * ldh + c] = c < sm.kk ? g / (1.0f + expf(-g)) * au[i][j] : 0.0f;
            }
        }
}

__global__ __launch_bounds__(256) void gemm2_f32_kernel(Gemm2Params<float> p) {
    __shared__ float As[BK][BM + 4];
    __shared__ float Bs[BK][BN + 4];
    int s, local;
    SegMeta sm;
    if (!tile_of(p, blockIdx.x, s, sm, local)) return;
    const int mt = ceil_div(sm.rows, BM);
    const int mtile = local % mt, ntile = local / mt;
    const bool shared = sm.e < 0;
    const float* Hb = shared ? p.Hs : p.H + (size_t)sm.row0 * p.I;
    const RoutedWeights rw = shared ? RoutedWeights{0, 0, p.Is} : routed_weights(p, sm);
    const int ldh = shared ? p.Is : p.I;  // H row stride
    const float* Wd = shared ? p.sd : p.wd + rw.base;
    const int K = sm.kg;

    const int tid = threadIdx.x;
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    const int row = mtile * BM + lr;
    const float* asrc = row < sm.rows ? Hb + (size_t)row * ldh : nullptr;
    const int n = ntile * BN + lr;
    const float* bsrc = n < p.d ? Wd + (size_t)n * rw.ldd : nullptr;

    const int ty = tid >> 4, tx = tid & 15;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += BK) {
        const int kb = k0 + lk;
        float a[4] = {0.f, 0.f, 0.f, 0.f}, b[4] = {0.f, 0.f, 0.f, 0.f};
        if (kb < K) {  // kb % 4 == 0 and the strides are multiples of 8: the vector is in bounds
            const float4 va = asrc ? *reinterpret_cast<const float4*>(asrc + kb) : make_float4(0.f, 0.f, 0.f, 0.f);
            const float4 vb = bsrc ? *reinterpret_cast<const float4*>(bsrc + kb) : make_float4(0.f, 0.f, 0.f, 0.f);
            a[0] = va.x; a[1] = va.y; a[2] = va.z; a[3] = va.w;
            b[0] = vb.x; b[1] = vb.y; b[2] = vb.z; b[3] = vb.w;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (kb + q >= K) a[q] = b[q] = 0.f;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            As[lk + q][lr] = a[q];
            Bs[lk + q][lr] = b[q];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < BK; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
    float* Ob = shared ? p.Os : p.O + (size_t)sm.row0 * p.d;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = mtile * BM + ty * 4 + i;
            const int c = ntile * BN + tx * 4 + j;
            if (r < sm.rows && c < p.d) Ob[(size_t)r * p.d + c] = acc[i][j];
        }
}

hipError_t launch_gemm1_f32(const Gemm1Params<float>& p, int grid, hipStream_t s) {
    if (grid <= 0) return hipSuccess;
    gemm1_f32_kernel<<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_gemm2_f32(const Gemm2Params<float>& p, int grid, hipStream_t s) {
    if (grid <= 0) return hipSuccess;
    gemm2_f32_kernel<<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace flexmoe
