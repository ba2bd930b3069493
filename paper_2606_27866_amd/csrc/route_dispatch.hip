// Routing and token dispatch (FlexMoE App. C.3: the gather / sort-by-expert
// step of the kernelized clipped FFN, done on the device without host syncs).
//
//   route_kernel           top-k over fp32 logits + softmax weights, one wave
//                          per token, and the expert histogram of each chunk
//                          of kRouteTokens tokens
//   dispatch_scan_kernel   per expert, exclusive scan of the chunk histograms
//   dispatch_scatter_kernel  stable placement of every assignment into the
//                          expert-grouped order (ascending assignment id inside
//                          an expert), inverse map, segment and tile tables
//   dispatch_small_kernel  all three in one workgroup, for decode-sized T
//
// Experts with k_e = 0 are left out of the grouped order (pos = -1) but still
// counted.  Nothing here uses atomics whose arrival order could change a
// result: ranks come from wave ballots and scans, so the permutation is
// bit-reproducible, and both dispatch paths produce the same bits.
#include "kernels.h"

namespace flexmoe {

// Routing order: larger logit first, equal logits -> lower id, NaN last.
// route_key maps a logit to an unsigned key with the same order: the bits of
// a non-negative float with the sign bit set, those of a negative float
// inverted, -0 as +0 (they compare equal), and 0 for NaN (below -inf, whose
// key is 0x007fffff).  Expert a then comes before expert b exactly when
// key_a > key_b, or key_a == key_b and a < b.
__device__ __forceinline__ uint32_t route_key(float v) {
    uint32_t u = __float_as_uint(v);
    u = u == 0x80000000u ? 0u : u;
    const uint32_t k = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return __builtin_isnan(v) ? 0u : k;
}

// Per-wave LDS scratch of route_token: the token's keys and the k slots.
struct RouteScratch {
    uint32_t key[kMaxExperts];
    float slot_v[kMaxTopK];
    int slot_id[kMaxTopK];
};

// The logits of one token, experts lane + 64*q (q < 4), as four independent
// loads (addresses clamped into the row; entries past E are replaced by 0).
__device__ __forceinline__ void load_logits(const float* __restrict__ l, int E, int lane, float (&v)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane + 64 * q;
        const float t = l[min(e, E - 1)];
        v[q] = e < E ? t : 0.0f;
    }
}

// Ranks of this lane's experts lane + 64*q (q < NQ) among the E8 keys in LDS:
// the number of experts ordered before each.  Every lane reads the same keys
// (an LDS broadcast); two compares per pair, no branches.
template <int NQ>
__device__ __forceinline__ void rank_keys(const RouteScratch& rs, const uint32_t (&mk)[4], int E8, int lane,
                                          int (&rank)[4]) {
    for (int j0 = 0; j0 < E8; j0 += 8) {
        const uint4 k0 = *reinterpret_cast<const uint4*>(&rs.key[j0]);
        const uint4 k1 = *reinterpret_cast<const uint4*>(&rs.key[j0 + 4]);
        const uint32_t o[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int me = lane + 64 * q;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                rank[q] += (o[i] > mk[q]) + (o[i] == mk[q] && j0 + i < me);
        }
    }
}

// One wave routes one token whose logits are in v (load_logits): lane j < k
// returns the j-th selected expert and its router weight.  Each lane ranks
// its (up to four) experts by counting the experts ordered before them under
// the order above, reading the token's keys back from LDS.  Ranks are a
// permutation of 0..E-1, so the expert of rank j < k fills slot j -- the
// top-k in order, with no chain of cross-lane steps.  The LDS row is padded
// to a multiple of 8 with key 0 and ids at or past E, which no expert counts.
// Softmax over all E experts, shifted by the largest logit; with norm_topk
// the k weights are divided by their sum.
__device__ __forceinline__ void route_token(const float (&v)[4], int E, int k, int norm_topk, int lane,
                                            RouteScratch& rs, int& my_id, float& my_w) {
    const int nq = ceil_div(E, 64);         // wave-uniform
    const int E8 = ceil_div(E, 8) * 8;      // <= kMaxExperts
    uint32_t mk[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane + 64 * q;
        mk[q] = route_key(v[q]);
        if (e < E) rs.key[e] = mk[q];
        else if (e < E8) rs.key[e] = 0u;
    }
    __builtin_amdgcn_wave_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    int rank[4] = {0, 0, 0, 0};
    switch (nq) {
        case 1: rank_keys<1>(rs, mk, E8, lane, rank); break;
        case 2: rank_keys<2>(rs, mk, E8, lane, rank); break;
        case 3: rank_keys<3>(rs, mk, E8, lane, rank); break;
        default: rank_keys<4>(rs, mk, E8, lane, rank); break;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane + 64 * q;
        if (e < E && rank[q] < k) {
            rs.slot_id[rank[q]] = e;
            rs.slot_v[rank[q]] = v[q];
        }
    }
    __builtin_amdgcn_wave_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    const float m = rs.slot_v[0];
    my_id = lane < k ? rs.slot_id[lane] : 0;
    const float my_logit = lane < k ? rs.slot_v[lane] : 0.0f;
    __builtin_amdgcn_wave_barrier();  // the scratch is reused by the wave's next token
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    float z = 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (lane + 64 * q < E) z += expf(v[q] - m);
    z = wave_total_f(z);
    float w = lane < k ? expf(my_logit - m) / z : 0.0f;
    if (norm_topk) w = w / wave_total_f(w);
    my_w = w;
}

// One wave: exclusive scan over experts of the active counts (k_e > 0, k_e
// clamped to [0, I]; device data is never trusted for addressing), four
// experts per lane.  Also scans the packed widths of the clipped weight
// layout: an expert whose block would end past packed_limit is treated as
// k_e = 0.  Fills off[], kk_s[], ch0[] and zeroes run[]; returns P.
template <typename CountFn, typename KeepFn>
__device__ __forceinline__ int expert_offsets(CountFn count, KeepFn keep, int E, int I, int packed_limit,
                                              int* off, int* kk_s, int* ch0, int* run) {
    const int lane = threadIdx.x & 63;
    int k4[4], w4 = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane * 4 + q;
        k4[q] = e < E ? min(max(keep(e), 0), I) : 0;
        w4 += packed_width(k4[q]);
    }
    // packed channel offsets (a prefix of at most 256 * 2^20 fits in int)
    const int winc = wave_incl_scan(w4);
    int wbase = winc - w4;
    int c4[4], local = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane * 4 + q;
        const int w = packed_width(k4[q]);
        if (e < E) ch0[e] = wbase;
        if (wbase + w > packed_limit) k4[q] = 0;
        wbase += w;
        c4[q] = (e < E && k4[q] > 0) ? count(e) : 0;
        local += c4[q];
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
        } else {
            kk_s[e] = -1;  // below every width: the down-order ranking counts no such entry
        }
        base += c4[q];
    }
    return lane63(inc);
}

// One wave: segment table (shared expert first: its tiles carry the longest
// reductions, so they start first), the exclusive scan of the gate/up GEMM's
// tile counts in segment order, and the down GEMM's tile order (order2, see
// Gemm2Params::order) with its tile counts scanned in that order, 64
// segments per round.  n2s and ordl are LDS scratch of nseg entries.
// rank(e): the number of experts ordered before expert e (see below).
template <typename CountFn, typename RankFn>
__device__ void write_tables(CountFn count, RankFn rank, const int* off, const int* kk_s, const int* ch0,
                             const int32_t* __restrict__ plan, int P, int T, int E, int I,
                             int I_shared, int d, TileShape ts, int* n2s, int* ordl,
                             int32_t* __restrict__ offsets, SegMeta* __restrict__ seg,
                             int32_t* __restrict__ t1start, int32_t* __restrict__ t2start,
                             int32_t* __restrict__ order2) {
    const int lane = threadIdx.x & 63;
    const int hs = I_shared > 0 ? 1 : 0;
    const int nseg = E + hs;
    int c1 = 0, c3 = 0, c4 = 0;
    for (int s0 = 0; s0 < nseg; s0 += 64) {
        const int s = s0 + lane;
        int n1 = 0, n2 = 0, n3 = 0, n4 = 0;
        SegMeta m{};
        if (s < nseg) {
            if (s < hs) {
                m.row0 = 0;
                m.rows = T;
                m.kk = I_shared;
                m.ch0 = 0;
                m.kg = I_shared;
                m.e = -1;
            } else {
                // plan entries are device data: clamped so that addressing stays in range
                const int e = plan ? min(max(plan[s - hs], 0), E - 1) : s - hs;
                m.row0 = off[e];
                m.rows = kk_s[e] > 0 ? count(e) : 0;
                m.kk = kk_s[e];
                m.ch0 = ch0[e];
                m.kg = plan && m.kk > 0 ? min(max(plan[E + e], m.kk), I) : m.kk;
                m.e = e;
                n3 = packed_width(m.rows);
                n4 = ceil_div(m.rows, ts.bm1);
            }
            if (m.rows > 0 && m.kk > 0) {
                n1 = ceil_div(m.rows, ts.bm1) * ceil_div(m.kg, ts.bn1);
                n2 = ceil_div(m.rows, ts.bm2) * ceil_div(d, ts.bn2);
                if (s < hs && ts.ks2 > 0) n2 *= ceil_div(m.kk, ts.ks2);
            }
            n2s[s] = n2;
        }
        if (s >= hs && s < nseg) offsets[s - hs] = off[s - hs];
        const int i1 = wave_incl_scan(n1);
        const int i3 = wave_incl_scan(n3), i4 = wave_incl_scan(n4);
        if (s < nseg) {
            t1start[s] = c1 + i1 - n1;
            m.prow0 = s < hs ? 0 : c3 + i3 - n3;
            m.rt0 = s < hs ? 0 : c4 + i4 - n4;
            seg[s] = m;
        }
        c1 += lane63(i1);
        c3 += lane63(i3);
        c4 += lane63(i4);
    }
    // The down GEMM's tile order: the shared expert, then the routed experts
    // by decreasing width k_e (ties: lower id first), so that the longest
    // reductions are handed out first.  The bucketed forward keeps its
    // plan's order (one launch per width group).
    if (hs && lane == 0) {
        ordl[0] = 0;
        order2[0] = 0;
    }
    for (int e0 = 0; e0 < E; e0 += 64) {
        const int e = e0 + lane;
        if (e >= E) continue;
        const int pos = plan ? e : rank(e);
        ordl[hs + pos] = hs + e;
        order2[hs + pos] = hs + e;
    }
    __builtin_amdgcn_wave_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    int c2 = 0;
    for (int i0 = 0; i0 < nseg; i0 += 64) {
        const int i = i0 + lane;
        const int n2 = i < nseg ? n2s[ordl[i]] : 0;
        const int i2 = wave_incl_scan(n2);
        if (i < nseg) t2start[i] = c2 + i2 - n2;
        c2 += lane63(i2);
    }
    if (lane == 0) {
        offsets[E] = P;
        t1start[nseg] = c1;
        t2start[nseg] = c2;
    }
}

// Expert e's place in the down GEMM's order counts the experts ordered
// before it: wider ones, and equal widths with a lower id.  width_rank4 adds
// the experts q0 .. q0+3, read as one 16-byte LDS access (kk_s is 16-byte
// aligned and holds kMaxExperts entries; entries at or past E hold -1, which
// no width is below, so the count needs no bound check).
static_assert(kMaxExperts == 4 * 64, "expert_offsets fills all of kk_s (four entries per lane)");
__device__ __forceinline__ int width_rank4(const int* kk_s, int q0, int ks, int e) {
    const int4 v = *reinterpret_cast<const int4*>(&kk_s[q0]);
    return (v.x > ks) + (v.x == ks && q0 < e) + (v.y > ks) + (v.y == ks && q0 + 1 < e) + (v.z > ks) +
           (v.z == ks && q0 + 2 < e) + (v.w > ks) + (v.w == ks && q0 + 3 < e);
}

// One wave: stable placement of assignments [a0, a1) in rounds of 64.  The
// match mask of equal expert ids comes from 8 ballots; a lane's rank is the
// number of matching lower lanes; the lowest matching lane advances run[e].
// base(e) is where this range's first assignment of expert e goes.
template <typename BaseFn>
__device__ __forceinline__ void place(const int32_t* __restrict__ idx, int a0, int a1, const int* kk_s,
                                      int* run, BaseFn base, int32_t* __restrict__ perm,
                                      int32_t* __restrict__ pos) {
    const int lane = threadIdx.x & 63;
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
        __builtin_amdgcn_wave_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        if (valid) {
            if (kk_s[e] > 0) {
                const int dst = base(e) + r + rank;
                perm[dst] = a;
                pos[a] = dst;
            } else {
                pos[a] = -1;
            }
            if ((match & lt) == 0) run[e] = r + __popcll(match);
        }
        __builtin_amdgcn_wave_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
    }
}

// One chunk of kRouteTokens tokens per workgroup, one wave per token.
__global__ __launch_bounds__(64 * kRouteTokens) void route_kernel(
    const float* __restrict__ logits, int T, int E, int k, int norm_topk,
    int32_t* __restrict__ idx, float* __restrict__ wts, int32_t* __restrict__ blockcnt, int NB) {
    __shared__ int hist[kMaxExperts];
    __shared__ RouteScratch rs[kRouteTokens];
    for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
    __syncthreads();
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int t = blockIdx.x * kRouteTokens + wave;
    if (t < T) {  // uniform across the wave
        int id;
        float w, v[4];
        load_logits(logits + (size_t)t * E, E, lane, v);
        route_token(v, E, k, norm_topk, lane, rs[wave], id, w);
        if (lane < k) {
            idx[(size_t)t * k + lane] = id;
            wts[(size_t)t * k + lane] = w;
            atomicAdd(&hist[id], 1);  // a count: arrival order does not matter
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

__global__ __launch_bounds__(64) void dispatch_scatter_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ keep,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ blockbase, int T, int E, int k,
    int I, int I_shared, int d, int NB, TileShape ts, int packed_limit, const int32_t* __restrict__ plan,
    int32_t* __restrict__ perm,
    int32_t* __restrict__ pos, int32_t* __restrict__ offsets, SegMeta* __restrict__ seg,
    int32_t* __restrict__ t1start, int32_t* __restrict__ t2start, int32_t* __restrict__ order2) {
    __shared__ int off[kMaxExperts];
    __shared__ __align__(16) int kk_s[kMaxExperts];
    __shared__ int ch0[kMaxExperts];
    __shared__ int run[kMaxExperts];
    __shared__ int n2s[kMaxExperts + 1];
    __shared__ int ordl[kMaxExperts + 1];
    auto count = [&](int e) { return counts[e]; };
    auto keep_of = [&](int e) { return keep[e]; };
    const int P = expert_offsets(count, keep_of, E, I, packed_limit, off, kk_s, ch0, run);
    __syncthreads();
    if (blockIdx.x == 0) {
        auto rank = [&](int e) {
            const int ks = kk_s[e];
            int r = 0;
#pragma unroll 4
            for (int q0 = 0; q0 < E; q0 += 4) r += width_rank4(kk_s, q0, ks, e);
            return r;
        };
        write_tables(count, rank, off, kk_s, ch0, plan, P, T, E, I, I_shared, d, ts, n2s, ordl, offsets, seg,
                     t1start, t2start, order2);
    }
    const int a0 = blockIdx.x * kRouteTokens * k;
    const int a1 = min((blockIdx.x + 1) * kRouteTokens, T) * k;
    auto base = [&](int e) { return off[e] + blockbase[(size_t)e * NB + blockIdx.x]; };
    place(idx, a0, a1, kk_s, run, base, perm, pos);
}

// Route, count, scan and place in one workgroup (T * k <= kSmallAssign).
// Wave w routes the contiguous tokens [w*per, (w+1)*per) and counts its own
// expert histogram; a scan over the waves gives each wave its base inside
// every expert's segment, so the 16 waves place their assignments at once,
// in the same order as one pass over the tokens would.  With pre_routed the
// tokens were routed by route_kernel (spread over several compute units):
// the waves read their tokens' expert ids instead.
__global__ __launch_bounds__(64 * kSmallWaves) void dispatch_small_kernel(
    const float* __restrict__ logits, int T, int E, int k, int norm_topk,
    const int32_t* __restrict__ keep, int I, int I_shared, int d, TileShape ts, int packed_limit,
    const int32_t* __restrict__ plan, int pre_routed, int32_t* __restrict__ idx, float* __restrict__ wts,
    int32_t* __restrict__ counts,
    int32_t* __restrict__ perm, int32_t* __restrict__ pos, int32_t* __restrict__ offsets,
    SegMeta* __restrict__ seg, int32_t* __restrict__ t1start, int32_t* __restrict__ t2start,
    int32_t* __restrict__ order2) {
    __shared__ int hist[kSmallWaves][kMaxExperts];  // per-wave counts, then per-wave bases
    __shared__ int cnt[kMaxExperts];
    __shared__ int off[kMaxExperts];
    __shared__ __align__(16) int kk_s[kMaxExperts];
    __shared__ int ch0[kMaxExperts];
    __shared__ int run[kMaxExperts];
    __shared__ int n2s[kMaxExperts + 1];
    __shared__ int ordl[kMaxExperts + 1];
    __shared__ int32_t sidx[kSmallAssign];
    __shared__ RouteScratch rs[kSmallWaves];
    __shared__ int keep_s[kMaxExperts];
    __shared__ int part[kSmallWaves][kMaxExperts];  // per-wave partial counts of the width ranks
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    for (int e = lane; e < E; e += 64) hist[wave][e] = 0;
    // the budget is read while the first wave routes
    if (wave == kSmallWaves - 1)
        for (int e = lane; e < E; e += 64) keep_s[e] = keep[e];
    __builtin_amdgcn_wave_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    const int per = ceil_div(T, kSmallWaves);
    const int t0 = min(T, wave * per), t1 = min(T, t0 + per);
    if (pre_routed) {
        for (int a = t0 * k + lane; a < t1 * k; a += 64) {
            const int id = min(max(idx[a], 0), E - 1);
            sidx[a] = id;
            atomicAdd(&hist[wave][id], 1);  // a count: arrival order does not matter
        }
    }
    // the next token's logits are loaded while this one is ranked
    float vn[4];
    if (!pre_routed && t0 < t1) load_logits(logits + (size_t)t0 * E, E, lane, vn);
    for (int t = pre_routed ? t1 : t0; t < t1; ++t) {
        int id;
        float w, v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = vn[q];
        if (t + 1 < t1) load_logits(logits + (size_t)(t + 1) * E, E, lane, vn);
        route_token(v, E, k, norm_topk, lane, rs[wave], id, w);
        if (lane < k) {
            idx[(size_t)t * k + lane] = id;
            wts[(size_t)t * k + lane] = w;
            sidx[t * k + lane] = id;
            atomicAdd(&hist[wave][id], 1);  // a count: arrival order does not matter
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        int c = 0;
        for (int w = 0; w < kSmallWaves; ++w) {
            const int h = hist[w][e];
            hist[w][e] = c;
            c += h;
        }
        cnt[e] = c;
        counts[e] = c;
    }
    __syncthreads();
    auto count = [&](int e) { return cnt[e]; };
    int P = 0;
    if (wave == 0) {
        auto keep_of = [&](int e) { return keep_s[e]; };
        P = expert_offsets(count, keep_of, E, I, packed_limit, off, kk_s, ch0, run);
    }
    __syncthreads();
    // the down GEMM's order: every wave counts, for each expert, the experts
    // of its share of the width table ordered before it (wave w: entries 4w
    // .. 4w+3, then 64 further on, ...); the first wave adds the shares
    if (!plan) {
        for (int e0 = 0; e0 < E; e0 += 64) {
            const int e = e0 + lane;
            const int ks = kk_s[min(e, kMaxExperts - 1)];
            int r = 0;
            for (int q0 = wave * 4; q0 < E; q0 += kSmallWaves * 4) r += width_rank4(kk_s, q0, ks, e);
            if (e < E) part[wave][e] = r;
        }
    }
    __syncthreads();
    if (wave == 0) {
        auto rank = [&](int e) {
            int r = 0;
#pragma unroll
            for (int w = 0; w < kSmallWaves; ++w) r += part[w][e];
            return r;
        };
        write_tables(count, rank, off, kk_s, ch0, plan, P, T, E, I, I_shared, d, ts, n2s, ordl, offsets, seg,
                     t1start, t2start, order2);
    }
    __syncthreads();
    // this wave's running position inside each expert starts at its base
    auto base = [&](int e) { return off[e]; };
    place(sidx, t0 * k, t1 * k, kk_s, hist[wave], base, perm, pos);
}

__global__ void set_keep_kernel(int32_t* __restrict__ keep, KeepArgs t, int E) {
    const int e = threadIdx.x;
    if (e < E) keep[e] = t.v[e];
}

__global__ void set_plan_kernel(int32_t* __restrict__ keep, int32_t* __restrict__ plan, KeepArgs k,
                                KeepArgs order, KeepArgs kg, int E) {
    const int e = threadIdx.x;
    if (e < E) {
        keep[e] = k.v[e];
        plan[e] = order.v[e];
        plan[E + e] = kg.v[e];
    }
}

}  // namespace flexmoe
