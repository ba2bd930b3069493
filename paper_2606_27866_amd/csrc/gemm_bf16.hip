// Ragged grouped GEMMs of the masked expert FFN on bf16 MFMA (gfx950).
//
// gemm1: for every segment s (a routed expert with k_s = k_e channels, or the
//   shared expert) and every row routed to it, the gate and up projections of
//   the first k_s ranked channels (Eq. 4) and SwiGLU in registers:
//     H[row][c] = silu(<W_gate[c], x>) * <W_up[c], x>     c < k_s
//   The channel extent of a segment's tile grid is ceil(k_s / BN): pruned
//   channels are neither loaded nor multiplied.  Gate and up tiles of the
//   same channels are held side by side in LDS so both accumulators of a
//   channel sit in the same lanes (no gate/up interleaving of the weights).
// gemm2: the down projection with the reduction extent truncated to k_s:
//     O[row][n] = sum_{c < k_s} H[row][c] * W_down[n][c]
//
// Both operands are K-contiguous in memory ([rows][K]), tiles are staged
// through LDS with register double buffering, and each wave accumulates a
// 64 x 64 (gemm1: 64 rows x 32 channels x {gate, up}) block with
// v_mfma_f32_16x16x32_bf16 in fp32.  Tiles come from the device-built tile
// table (segment-major, row tiles fastest), so the host never learns the
// routing.
#include "kernels.h"

namespace flexmoe {

namespace {
constexpr int BK = 64;
constexpr int LDSW = BK + 8;   // padded LDS row (elements): 144 B per row

__device__ __forceinline__ bf16x8 lds_frag(const bf16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}
}  // namespace

__global__ __launch_bounds__(256) void gemm1_bf16_kernel(Gemm1Params<bf16_t> p) {
    constexpr int BM = kBf16BM1, BN = kBf16BN1;
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDSW];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][2 * BN * LDSW];

    const int L = blockIdx.x;
    if (L >= p.tstart[p.nseg]) return;
    const int s = find_segment(p.tstart, p.nseg, L);
    const SegMeta sm = p.seg[s];
    const int local = L - p.tstart[s];
    const int mt = ceil_div(sm.rows, BM);
    const int mtile = local % mt, ntile = local / mt;
    const int hs = p.nseg - p.E;  // 1 if segment 0 is the shared expert
    const bool shared = s < hs;
    const size_t wofs = shared ? 0 : (size_t)(s - hs) * p.I * p.d;
    const bf16_t* Wg = (shared ? p.sg : p.wg) + wofs;
    const bf16_t* Wu = (shared ? p.su : p.wu) + wofs;

    const int tid = threadIdx.x;
    const int lr = tid >> 3;        // 0..31
    const int lc = (tid & 7) * 8;   // element offset inside the K tile
    const bf16_t* asrc[4];
    const bf16_t* bsrc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = lr + 32 * j;
        const int row = mtile * BM + r;
        asrc[j] = nullptr;
        if (row < sm.rows) {
            // the clamp only guards memory if the caller rewrote the keep table
            // while this forward was in flight; consistent inputs never need it
            const int t = shared ? row : (int)min((unsigned)(p.perm[sm.row0 + row] / p.top_k), (unsigned)(p.tokens - 1));
            asrc[j] = p.x + (size_t)t * p.d;
        }
        const int ch = ntile * BN + (r & (BN - 1));
        bsrc[j] = ch < sm.kk ? (r < BN ? Wg : Wu) + (size_t)ch * p.d : nullptr;
    }

    u32x4 ra[4], rb[4];
    const u32x4 zero = {0u, 0u, 0u, 0u};
    auto gload = [&](int k0) {
        const bool kin = k0 + lc < p.d;  // d % 8 == 0: a vector is all in or all out
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            ra[j] = (asrc[j] && kin) ? *reinterpret_cast<const u32x4*>(asrc[j] + k0 + lc) : zero;
            rb[j] = (bsrc[j] && kin) ? *reinterpret_cast<const u32x4*>(bsrc[j] + k0 + lc) : zero;
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            *reinterpret_cast<u32x4*>(&As[buf][(lr + 32 * j) * LDSW + lc]) = ra[j];
            *reinterpret_cast<u32x4*>(&Bs[buf][(lr + 32 * j) * LDSW + lc]) = rb[j];
        }
    };

    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave >> 1, wn = wave & 1;
    floatx4 accg[4][2], accu[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            accg[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
            accu[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        }

    const int nk = ceil_div(p.d, BK);
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            const int kof = ks * 32 + (lane >> 4) * 8;
            bf16x8 a[4], bg[2], bu[2];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                a[i] = lds_frag(&As[cur][(wm * 64 + i * 16 + (lane & 15)) * LDSW + kof]);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                bg[j] = lds_frag(&Bs[cur][(wn * 32 + j * 16 + (lane & 15)) * LDSW + kof]);
                bu[j] = lds_frag(&Bs[cur][(BN + wn * 32 + j * 16 + (lane & 15)) * LDSW + kof]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    accg[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bg[j], accg[i][j], 0, 0, 0);
                    accu[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bu[j], accu[i][j], 0, 0, 0);
                }
        }
        if (kt + 1 < nk) lstore(cur ^ 1);
        __syncthreads();
    }

    bf16_t* Hb = shared ? p.Hs : p.H + (size_t)sm.row0 * p.I;
    const int ldh = shared ? p.Is : p.I;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = mtile * BM + wm * 64 + i * 16 + (lane >> 4) * 4 + r;
                const int ch = ntile * BN + wn * 32 + j * 16 + (lane & 15);
                if (row < sm.rows && ch < sm.kk)
                    Hb[(size_t)row * ldh + ch] = f32_to_bf16(silu_fast(accg[i][j][r]) * accu[i][j][r]);
            }
}

__global__ __launch_bounds__(256) void gemm2_bf16_kernel(Gemm2Params<bf16_t> p) {
    constexpr int BM = kBf16BM2, BN = kBf16BN2;
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDSW];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN * LDSW];

    const int L = blockIdx.x;
    if (L >= p.tstart[p.nseg]) return;
    const int s = find_segment(p.tstart, p.nseg, L);
    const SegMeta sm = p.seg[s];
    const int local = L - p.tstart[s];
    const int mt = ceil_div(sm.rows, BM);
    const int mtile = local % mt, ntile = local / mt;
    const int hs = p.nseg - p.E;  // 1 if segment 0 is the shared expert
    const bool shared = s < hs;
    const bf16_t* Hb = shared ? p.Hs : p.H + (size_t)sm.row0 * p.I;
    const int ldh = shared ? p.Is : p.I;
    const bf16_t* Wd = shared ? p.sd : p.wd + (size_t)(s - hs) * p.d * p.I;
    const int K = sm.kk;

    const int tid = threadIdx.x;
    const int lr = tid >> 3;
    const int lc = (tid & 7) * 8;
    const bf16_t* asrc[4];
    const bf16_t* bsrc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = lr + 32 * j;
        const int row = mtile * BM + r;
        asrc[j] = row < sm.rows ? Hb + (size_t)row * ldh : nullptr;
        const int n = ntile * BN + r;
        bsrc[j] = n < p.d ? Wd + (size_t)n * ldh : nullptr;  // W_down rows have the H stride
    }

    u32x4 ra[4], rb[4];
    const u32x4 zero = {0u, 0u, 0u, 0u};
    auto gload = [&](int k0) {
        const int kb = k0 + lc;
        const int nv = K - kb;  // valid elements of this vector (row strides are multiples of 8)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            u32x4 va = zero, vb = zero;
            if (nv > 0) {
                if (asrc[j]) va = *reinterpret_cast<const u32x4*>(asrc[j] + kb);
                if (bsrc[j]) vb = *reinterpret_cast<const u32x4*>(bsrc[j] + kb);
                if (nv < 8) {
                    va = mask_tail_bf16(va, nv);
                    vb = mask_tail_bf16(vb, nv);
                }
            }
            ra[j] = va;
            rb[j] = vb;
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            *reinterpret_cast<u32x4*>(&As[buf][(lr + 32 * j) * LDSW + lc]) = ra[j];
            *reinterpret_cast<u32x4*>(&Bs[buf][(lr + 32 * j) * LDSW + lc]) = rb[j];
        }
    };

    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave >> 1, wn = wave & 1;
    floatx4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int nk = ceil_div(K, BK);
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            const int kof = ks * 32 + (lane >> 4) * 8;
            bf16x8 a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                a[i] = lds_frag(&As[cur][(wm * 64 + i * 16 + (lane & 15)) * LDSW + kof]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                b[j] = lds_frag(&Bs[cur][(wn * 64 + j * 16 + (lane & 15)) * LDSW + kof]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) lstore(cur ^ 1);
        __syncthreads();
    }

    float* Ob = shared ? p.Os : p.O + (size_t)sm.row0 * p.d;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = mtile * BM + wm * 64 + i * 16 + (lane >> 4) * 4 + r;
                const int n = ntile * BN + wn * 64 + j * 16 + (lane & 15);
                if (row < sm.rows && n < p.d) Ob[(size_t)row * p.d + n] = acc[i][j][r];
            }
}

hipError_t launch_gemm1_bf16(const Gemm1Params<bf16_t>& p, int grid, hipStream_t s) {
    if (grid <= 0) return hipSuccess;
    gemm1_bf16_kernel<<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_gemm2_bf16(const Gemm2Params<bf16_t>& p, int grid, hipStream_t s) {
    if (grid <= 0) return hipSuccess;
    gemm2_bf16_kernel<<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace flexmoe
