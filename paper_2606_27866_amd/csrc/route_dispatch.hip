// Routing and token dispatch (FlexMoE App. C.3: the gather / sort-by-expert
// step of the kernelized clipped FFN, done on the device without host syncs).
//
//   route_kernel           top-k over fp32 logits + softmax weights, and a
//                          per-chunk expert histogram (chunk = 64 tokens)
//   dispatch_scan_kernel   per expert, exclusive scan of the chunk histogram
//   dispatch_scatter_kernel  stable placement of every assignment into the
//                          expert-grouped order (ascending assignment id inside
//                          an expert), inverse map, segment and tile tables
//
// Experts with k_e = 0 are left out of the grouped order (pos = -1) but still
// counted.  Nothing here uses atomics whose arrival order could change a
// result: ranks come from wave ballots and per-chunk scans, so the
// permutation is bit-reproducible.
#include "kernels.h"

namespace flexmoe {

// Routing order: larger logit first, equal logits -> lower id, NaN last.
__device__ __forceinline__ bool route_before(float va, int ia, float vb, int ib) {
    const bool na = __builtin_isnan(va), nb = __builtin_isnan(vb);
    if (na != nb) return nb;
    if (!na && va != vb) return va > vb;
    return ia < ib;
}

// One chunk of kRouteTokens tokens per workgroup, one wave per token.
constexpr int kRouteWaves = kRouteTokens;
constexpr int kTokPerWave = 1;

__global__ __launch_bounds__(64 * kRouteWaves) void route_kernel(
    const float* __restrict__ logits, int T, int E, int k, int norm_topk,
    int32_t* __restrict__ idx, float* __restrict__ wts, int32_t* __restrict__ blockcnt, int NB) {
    __shared__ int hist[kMaxExperts];
    for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int t0 = blockIdx.x * kRouteTokens + wave;
    float v[kTokPerWave][4];
#pragma unroll
    for (int i = 0; i < kTokPerWave; ++i) {
        const int t = t0 + i * kRouteWaves;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + 64 * q;
            v[i][q] = (t < T && e < E) ? logits[(size_t)t * E + e] : 0.0f;
        }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kTokPerWave; ++i) {
        const int t = t0 + i * kRouteWaves;
        if (t >= T) break;  // uniform across the wave
        bool taken[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) taken[q] = lane + 64 * q >= E;
        int my_id = 0;
        float my_logit = 0.0f, m = 0.0f;
        for (int j = 0; j < k; ++j) {
            float bv = 0.0f;
            int bi = -1;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int e = lane + 64 * q;
                if (!taken[q] && (bi < 0 || route_before(v[i][q], e, bv, bi))) {
                    bv = v[i][q];
                    bi = e;
                }
            }
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) {
                const float ov = __shfl_xor(bv, o, 64);
                const int oi = __shfl_xor(bi, o, 64);
                if (oi >= 0 && (bi < 0 || route_before(ov, oi, bv, bi))) {
                    bv = ov;
                    bi = oi;
                }
            }
            // every lane now holds the same winner (a total order makes the
            // butterfly reduction lane-independent)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (bi == lane + 64 * q) taken[q] = true;
            if (lane == j) {
                my_id = bi;
                my_logit = bv;
            }
            if (j == 0) m = bv;
        }
        float z = 0.0f;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (lane + 64 * q < E) z += expf(v[i][q] - m);
        z = wave_sum_f(z);
        float w = lane < k ? expf(my_logit - m) / z : 0.0f;
        if (norm_topk) w = w / wave_sum_f(w);
        if (lane < k) {
            idx[(size_t)t * k + lane] = my_id;
            wts[(size_t)t * k + lane] = w;
            atomicAdd(&hist[my_id], 1);  // a count: arrival order does not matter
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) blockcnt[(size_t)e * NB + blockIdx.x] = hist[e];
}

// Per expert: exclusive scan of its chunk counts.  Thread i owns a run of
// consecutive chunks, so all loads are in flight together.
__global__ __launch_bounds__(256) void dispatch_scan_kernel(const int32_t* __restrict__ blockcnt,
                                                            int NB, int32_t* __restrict__ blockbase,
                                                            int32_t* __restrict__ counts) {
    constexpr int kPer = 16;  // chunks per thread per round
    __shared__ int wsum[4];
    __shared__ int carry;
    const int e = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int32_t* src = blockcnt + (size_t)e * NB;
    int32_t* dst = blockbase + (size_t)e * NB;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int b0 = 0; b0 < NB; b0 += 256 * kPer) {
        const int base = b0 + threadIdx.x * kPer;
        int v[kPer];
        int local = 0;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            v[i] = base + i < NB ? src[base + i] : 0;
            local += v[i];
        }
        const int inc = wave_incl_scan(local);
        if (lane == 63) wsum[wave] = inc;
        __syncthreads();
        int pre = carry;
        for (int w = 0; w < wave; ++w) pre += wsum[w];
        int run = pre + inc - local;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            if (base + i < NB) dst[base + i] = run;
            run += v[i];
        }
        __syncthreads();
        if (threadIdx.x == 255) carry = pre + inc;
        __syncthreads();
    }
    if (threadIdx.x == 0) counts[e] = carry;
}

// Exclusive scan of per-segment tile counts, 64 segments per round.
__device__ void scan_tiles(const SegMeta* seg_l, int nseg, int d, TileShape ts,
                           int32_t* t1start, int32_t* t2start) {
    const int lane = threadIdx.x & 63;
    int c1 = 0, c2 = 0;
    for (int s0 = 0; s0 < nseg; s0 += 64) {
        const int s = s0 + lane;
        int n1 = 0, n2 = 0;
        if (s < nseg) {
            const SegMeta m = seg_l[s];
            if (m.rows > 0 && m.kk > 0) {
                n1 = ceil_div(m.rows, ts.bm1) * ceil_div(m.kk, ts.bn1);
                n2 = ceil_div(m.rows, ts.bm2) * ceil_div(d, ts.bn2);
            }
        }
        const int i1 = wave_incl_scan(n1), i2 = wave_incl_scan(n2);
        if (s < nseg) {
            t1start[s] = c1 + i1 - n1;
            t2start[s] = c2 + i2 - n2;
        }
        c1 += __shfl(i1, 63, 64);
        c2 += __shfl(i2, 63, 64);
    }
    if (lane == 0) {
        t1start[nseg] = c1;
        t2start[nseg] = c2;
    }
}

__global__ __launch_bounds__(64) void dispatch_scatter_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ keep,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ blockbase, int T, int E, int k,
    int I, int I_shared, int d, int NB, TileShape ts, int32_t* __restrict__ perm,
    int32_t* __restrict__ pos, int32_t* __restrict__ offsets, SegMeta* __restrict__ seg,
    int32_t* __restrict__ t1start, int32_t* __restrict__ t2start) {
    __shared__ int off[kMaxExperts];
    __shared__ int kk_s[kMaxExperts];
    __shared__ int run[kMaxExperts];
    __shared__ SegMeta seg_l[kMaxExperts + 1];
    const int lane = threadIdx.x;

    // exclusive scan of the active counts over experts (4 experts per lane)
    int c4[4], k4[4], local = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane * 4 + q;
        int kk = 0, c = 0;
        if (e < E) {
            kk = min(max(keep[e], 0), I);  // device data is clamped, never trusted
            c = kk > 0 ? counts[e] : 0;
        }
        c4[q] = c;
        k4[q] = kk;
        local += c;
    }
    const int inc = wave_incl_scan(local);
    int base = inc - local;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane * 4 + q;
        if (e < E) {
            off[e] = base;
            kk_s[e] = k4[q];
            run[e] = 0;
        }
        base += c4[q];
    }
    const int P = __shfl(inc, 63, 64);
    __syncthreads();

    if (blockIdx.x == 0) {
        // segment order: the shared expert (if any) first, then experts 0..E-1;
        // its tiles carry the longest reductions, so they start first
        const int hs = I_shared > 0 ? 1 : 0;
        const int nseg = E + hs;
        for (int e = lane; e < E; e += 64) {
            offsets[e] = off[e];
            SegMeta m;
            m.row0 = off[e];
            m.rows = kk_s[e] > 0 ? counts[e] : 0;
            m.kk = kk_s[e];
            m.pad = 0;
            seg_l[hs + e] = m;
            seg[hs + e] = m;
        }
        if (lane == 0) {
            offsets[E] = P;
            if (hs) {
                SegMeta m;
                m.row0 = 0;
                m.rows = T;
                m.kk = I_shared;
                m.pad = 0;
                seg_l[0] = m;
                seg[0] = m;
            }
        }
        __syncthreads();
        scan_tiles(seg_l, nseg, d, ts, t1start, t2start);
    }

    // stable placement: rounds of 64 consecutive assignments of this chunk
    const int a0 = blockIdx.x * kRouteTokens * k;
    const int a1 = min((blockIdx.x + 1) * kRouteTokens, T) * k;
    const uint64_t lt = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
    for (int r0 = a0; r0 < a1; r0 += 64) {
        const int a = r0 + lane;
        const bool valid = a < a1;
        const int e = valid ? idx[a] : 0;
        uint64_t match = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
            const bool b = (e >> bit) & 1;
            const uint64_t bb = __ballot(valid && b);
            match &= b ? bb : ~bb;
        }
        const int rank = __popcll(match & lt);
        const int r = valid ? run[e] : 0;
        __syncthreads();
        if (valid) {
            if (kk_s[e] > 0) {
                const int dst = off[e] + blockbase[(size_t)e * NB + blockIdx.x] + r + rank;
                perm[dst] = a;
                pos[a] = dst;
            } else {
                pos[a] = -1;
            }
            if ((match & lt) == 0) run[e] = r + __popcll(match);
        }
        __syncthreads();
    }
}

__global__ void set_keep_kernel(int32_t* __restrict__ keep, KeepArgs t, int E) {
    const int e = threadIdx.x;
    if (e < E) keep[e] = t.v[e];
}

}  // namespace flexmoe
