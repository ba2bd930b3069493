// Host side of the FlexMoE C ABI: argument checks, workspace carving and the
// launch sequence of one masked MoE-layer forward (include/flexmoe.h).
//
//   route -> dispatch scan -> dispatch scatter -> gate/up GEMM -> down GEMM
//   -> combine
//
// Launches go to the caller's stream, except the shared expert's two GEMMs,
// which run on a side stream forked before routing and joined before the
// combine.  The host never reads routing results back: tile counts live on
// the device and the routed GEMM grids are sized by an upper bound computed
// from (T, E, I); surplus workgroups exit at once.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "flexmoe.h"
#include "kernels.h"
#include "saliency.h"
#include "train.h"

using namespace flexmoe;

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(FLEXMOE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

int check_desc(const flexmoe_layer_desc* D) {
    if (!D) return fail(FLEXMOE_EINVAL, "desc is NULL");
    if (D->dtype != FLEXMOE_F32 && D->dtype != FLEXMOE_BF16)
        return fail(FLEXMOE_EDTYPE, "dtype %d is neither FLEXMOE_F32 nor FLEXMOE_BF16", D->dtype);
    if (D->norm_topk != 0 && D->norm_topk != 1)
        return fail(FLEXMOE_EINVAL, "norm_topk must be 0 or 1 (got %d)", D->norm_topk);
    if (D->d < 8 || D->d % 8) return fail(FLEXMOE_ESHAPE, "d = %d must be a positive multiple of 8", D->d);
    if (D->I < 8 || D->I % 8) return fail(FLEXMOE_ESHAPE, "I = %d must be a positive multiple of 8", D->I);
    if (D->I_shared < 0 || D->I_shared % 8)
        return fail(FLEXMOE_ESHAPE, "I_shared = %d must be 0 or a positive multiple of 8", D->I_shared);
    if (D->E < 1 || D->E > kMaxExperts)
        return fail(FLEXMOE_ESHAPE, "E = %d outside [1, %d]", D->E, kMaxExperts);
    if (D->top_k < 1 || D->top_k > D->E || D->top_k > kMaxTopK)
        return fail(FLEXMOE_ESHAPE, "top_k = %d outside [1, min(E, %d)]", D->top_k, kMaxTopK);
    if (D->max_tokens < 0) return fail(FLEXMOE_ESHAPE, "max_tokens = %d is negative", D->max_tokens);
    if ((long long)D->E * packed_width(D->I) >= (1LL << 31))
        return fail(FLEXMOE_ESHAPE, "E * I must stay below 2^31 channels");
    // every row index and tile count below stays inside int32
    const long long A = (long long)D->max_tokens * D->top_k;
    if (A + D->max_tokens > (1LL << 30))
        return fail(FLEXMOE_ESHAPE, "max_tokens * (top_k + 1) exceeds 2^30");
    if (D->dtype == FLEXMOE_BF16) {
        // the prefill GEMMs address each operand block with 32-bit byte offsets
        const long long T = D->max_tokens, wide = std::max(D->I, D->I_shared);
        if (T * std::max<long long>(D->d, wide) >= (1LL << 30) || wide * D->d >= (1LL << 30))
            return fail(FLEXMOE_ESHAPE,
                        "bf16 operand blocks must stay below 2^30 elements (max_tokens * max(d, I, "
                        "I_shared) and max(I, I_shared) * d)");
    }
    return FLEXMOE_OK;
}

struct Layout {
    size_t idx, wts, blockcnt, blockbase, counts, offsets, perm, pos, seg, t1, t2, ord2, keep, plan, H, Hs, O, Os;
    size_t total;
};

int num_chunks(int T) { return ceil_div(T, kRouteTokens); }

// Upper bound on the number of row tiles of height bm over all routed
// segments: sum_e ceil(n_e/bm) <= ceil(A/bm) + E - 1, <= E*ceil(T/bm)
// because a token routes to an expert at most once, and <= A because every
// tile holds at least one row.
long long routed_row_tiles_ub(int T, int E, int k, int bm) {
    const long long A = (long long)T * k;
    const long long a = (A + bm - 1) / bm + E - 1;
    const long long b = (long long)E * ((T + bm - 1) / bm);
    return std::min(std::min(a, b), A);
}

// The shared expert's down reduction is split into chunks (each writing its
// own partial rows, added by the combine in chunk order) while its tiles alone
// cover fewer than half of MI355X's 256 compute units: ceil(256 / tiles)
// chunks of at least kMinSplitK channels.  Its reductions are the longest of
// the launch (I_s against the routed experts' k_e <= I), so without the split
// they set the end of the down GEMM whenever the routed tiles finish first.
// From half of the compute units on, the concurrent routed tiles fill the
// rest and one reduction is faster (Qwen1.5-MoE shape, 4096 tokens: 128
// shared tiles, 0.7-1.9 % per step against two chunks).
constexpr int kComputeUnits = 256;
constexpr int kMinSplitK = 1024;
// Waves of shared-expert gate/up tiles below which the shared expert runs on
// the side stream during prefill.
constexpr int kSideWaves = 4;

// Chunk width of the shared expert's split down reduction for T tokens, 0 for
// one reduction over I_shared.  Decode-sized batches (weight streaming) use
// chunks of I channels.
int shared_ks2(const flexmoe_layer_desc& D, int T) {
    if (D.I_shared <= 0 || D.dtype != FLEXMOE_BF16) return 0;
    // weight streaming: chunks of one routed expert's worth of channels, two
    // above kSharedSplit2T tokens, where the shared expert's wide down tiles
    // compete with the routed experts' (fewer, longer tiles measured 1.3-2 %
    // faster per step there, 0.4-0.9 % slower at 1 and 8 tokens)
    if (T <= kDecodeMaxT) return T > kSharedSplit2T ? std::min(2 * D.I, D.I_shared) : D.I;
    const long long sh_tiles = (long long)ceil_div(T, kBigBM2) * ceil_div(D.d, kBigBN2);
    if (2 * sh_tiles >= kComputeUnits) return 0;
    const long long p = std::min<long long>(ceil_div(kComputeUnits, (int)sh_tiles), D.I_shared / kMinSplitK);
    if (p <= 1) return 0;
    return ceil_div(ceil_div(D.I_shared, (int)p), 64) * 64;
}

// Row sets of shared-expert output the combine adds (0 without a shared expert).
int shared_parts(const flexmoe_layer_desc& D, int T) {
    if (D.I_shared <= 0) return 0;
    const int ks2 = shared_ks2(D, T);
    return ks2 > 0 ? ceil_div(D.I_shared, ks2) : 1;
}

// Rows of the Os buffer a workspace for up to T tokens must hold: the largest
// shared_parts(T') * T' over T' <= T.  Splits happen only while the shared
// expert has fewer than kComputeUnits tiles, so the scan stops there.
size_t os_rows_bound(const flexmoe_layer_desc& D, int T) {
    if (D.I_shared <= 0 || T <= 0) return 0;
    size_t best = (size_t)T * shared_parts(D, T);
    // decode-sized batches: the chunk width depends on T
    for (int t = 1; t <= std::min(T, kDecodeMaxT); ++t) best = std::max(best, (size_t)t * shared_parts(D, t));
    const long long nd = ceil_div(D.d, kBigBN2);
    const long long t_end = std::min<long long>(T, (kComputeUnits + nd - 1) / nd * kBigBM2);
    for (long long t = kDecodeMaxT + 1; t <= t_end; ++t)
        best = std::max(best, (size_t)t * shared_parts(D, (int)t));
    return best;
}

Layout layout(const flexmoe_layer_desc& D, int T, size_t os_rows) {
    const size_t A = (size_t)T * D.top_k;
    const size_t NB = (size_t)num_chunks(T);
    const size_t nseg = (size_t)D.E + (D.I_shared > 0 ? 1 : 0);
    const size_t es = D.dtype == FLEXMOE_BF16 ? 2 : 4;
    Layout L{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off += align256(bytes);
        return o;
    };
    L.idx = take(A * 4);
    L.wts = take(A * 4);
    L.blockcnt = take((size_t)D.E * NB * 4);
    L.blockbase = take((size_t)D.E * NB * 4);
    L.counts = take((size_t)D.E * 4);
    L.offsets = take(((size_t)D.E + 1) * 4);
    L.perm = take(A * 4);
    L.pos = take(A * 4);
    L.seg = take(nseg * sizeof(SegMeta));
    L.t1 = take((nseg + 1) * 4);
    L.t2 = take((nseg + 1) * 4);
    L.ord2 = take(nseg * 4);
    L.keep = take((size_t)D.E * 4);      // bucketed forward: the uploaded keep table
    L.plan = take((size_t)D.E * 2 * 4);  // bucketed forward: segment order, GEMM widths
    L.H = take(A * (size_t)D.I * es);
    L.Hs = take((size_t)T * D.I_shared * es);
    const size_t os_es = D.dtype == FLEXMOE_BF16 ? 2 : 4;  // O / Os element size
    L.O = take(A * (size_t)D.d * os_es);
    // shared-expert rows, one row set per reduction chunk; last, so that the
    // offsets above depend on T alone
    L.Os = take(os_rows * D.d * os_es);
    L.total = off;
    return L;
}

// ---- optional per-kernel event timing --------------------------------------
struct TimedLaunch {
    int kernel;
    hipEvent_t start, stop;
};
std::mutex g_tmu;
bool g_timing = false;
std::vector<TimedLaunch> g_pending;
std::vector<hipEvent_t> g_free_events;
double g_ms[FLEXMOE_K_COUNT];
int64_t g_launches[FLEXMOE_K_COUNT];

hipEvent_t take_event() {
    if (!g_free_events.empty()) {
        hipEvent_t e = g_free_events.back();
        g_free_events.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Brackets one kernel launch with an event pair when timing is on.
struct KernelTimer {
    int kernel;
    hipStream_t s;
    hipEvent_t a = nullptr, b = nullptr;
    KernelTimer(int k, hipStream_t st) : kernel(k), s(st) {
        std::lock_guard<std::mutex> g(g_tmu);
        if (!g_timing) return;
        a = take_event();
        b = take_event();
        if (a && b) (void)hipEventRecord(a, s);
    }
    ~KernelTimer() {
        if (!a || !b) return;
        (void)hipEventRecord(b, s);
        std::lock_guard<std::mutex> g(g_tmu);
        g_pending.push_back({kernel, a, b});
    }
};

// ---- the side stream of the shared expert -------------------------------
// The shared expert's GEMMs need no routing, so they run on a second stream
// of the same device, forked from the caller's stream before routing starts
// and joined before the combine.  Its tiles then fill the compute units the
// routed GEMMs leave idle (their tails, the routing kernels).  One stream
// and two events per device are created on first use (default priority,
// non-blocking) and kept for the life of the process; the mutex keeps the
// fork/join of concurrent callers on one device apart.
struct SideStream {
    hipStream_t stream = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
    std::mutex mu;
};
constexpr int kMaxDevices = 64;
SideStream g_side[kMaxDevices];
std::mutex g_side_init;

int side_stream(SideStream** out) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return hip_fail(err, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(FLEXMOE_EHIP, "device %d beyond %d", dev, kMaxDevices);
    SideStream& ss = g_side[dev];
    std::lock_guard<std::mutex> g(g_side_init);
    if (!ss.stream) {
        hipStream_t st = nullptr;
        hipEvent_t a = nullptr, b = nullptr;
        if ((err = hipStreamCreateWithFlags(&st, hipStreamNonBlocking)) != hipSuccess)
            return hip_fail(err, "side stream create");
        // The fork and join events only order the two streams' kernels on
        // this device: nothing on the host or on another device waits for
        // them, so they skip the system-scope fence (a cache writeback and
        // invalidate at every record); each kernel's own end-of-kernel
        // release keeps its writes visible device-wide.  Decode steps run
        // 1-2.5 % faster.
        constexpr unsigned kEvFlags = hipEventDisableTiming | hipEventDisableSystemFence;
        if ((err = hipEventCreateWithFlags(&a, kEvFlags)) != hipSuccess ||
            (err = hipEventCreateWithFlags(&b, kEvFlags)) != hipSuccess) {
            (void)hipStreamDestroy(st);
            if (a) (void)hipEventDestroy(a);
            return hip_fail(err, "side stream event create");
        }
        ss.fork = a;
        ss.join = b;
        ss.stream = st;
    }
    *out = &ss;
    return FLEXMOE_OK;
}

// ---- scratch of the no-allocation forward --------------------------------
// flexmoe_layer_forward_noalloc takes its workspace from this file-scope
// device array instead of a caller buffer.  Every device the library runs
// on holds its own copy (64 MiB) from the module's load until the process
// ends.  In host code `scratch` names a host-side stand-in, not device
// memory: kernels and copies get the array's device address, looked up once
// per device with hipGetSymbolAddress (with that device current) and kept in
// g_scratch.
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];
void* g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

int scratch_address(void** out) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return hip_fail(err, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(FLEXMOE_EHIP, "device %d beyond %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* ptr = nullptr;
        err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return hip_fail(err, "hipGetSymbolAddress(scratch)");
        if (!ptr || ((uintptr_t)ptr & 255)) return fail(FLEXMOE_EHIP, "scratch address %p is not 256-byte aligned", ptr);
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return FLEXMOE_OK;
}

}  // namespace

extern "C" {

int flexmoe_timing_enable(int on) {
    std::lock_guard<std::mutex> g(g_tmu);
    g_timing = on != 0;
    if (g_timing) {
        for (int i = 0; i < FLEXMOE_K_COUNT; ++i) g_ms[i] = 0.0, g_launches[i] = 0;
    }
    return FLEXMOE_OK;
}

int flexmoe_timing_read(flexmoe_kernel_times* out) {
    if (!out) return fail(FLEXMOE_EINVAL, "timing_read: out is NULL");
    std::lock_guard<std::mutex> g(g_tmu);
    for (const TimedLaunch& t : g_pending) {
        hipError_t err = hipEventSynchronize(t.stop);
        float ms = 0.f;
        if (err == hipSuccess) err = hipEventElapsedTime(&ms, t.start, t.stop);
        if (err != hipSuccess) return hip_fail(err, "timing_read");
        g_ms[t.kernel] += ms;
        g_launches[t.kernel] += 1;
        g_free_events.push_back(t.start);
        g_free_events.push_back(t.stop);
    }
    g_pending.clear();
    for (int i = 0; i < FLEXMOE_K_COUNT; ++i) {
        out->ms[i] = g_ms[i];
        out->launches[i] = g_launches[i];
        g_ms[i] = 0.0;
        g_launches[i] = 0;
    }
    return FLEXMOE_OK;
}

const char* flexmoe_last_error(void) { return g_err; }

int flexmoe_keep_from_ratio(double r, int32_t I) {
    if (!(r >= 0.0 && r <= 1.0) || I < 1) {
        fail(FLEXMOE_EINVAL, "ratio %g outside [0, 1] or I = %d < 1", r, I);
        return -1;
    }
    double k = std::ceil(r * (double)I - 1e-9);
    if (k < 0) k = 0;
    if (k > I) k = I;
    return (int)k;
}

size_t flexmoe_workspace_bytes(const flexmoe_layer_desc* desc, int32_t T) {
    if (check_desc(desc) != FLEXMOE_OK) return 0;
    if (T < 0 || T > desc->max_tokens) {
        fail(FLEXMOE_ESHAPE, "T = %d outside [0, max_tokens = %d]", T, desc->max_tokens);
        return 0;
    }
    return layout(*desc, T, os_rows_bound(*desc, T)).total;
}

int flexmoe_set_budget(const flexmoe_layer_desc* desc, int32_t* keep_dev, const int32_t* keep_host,
                       void* stream) {
    int rc = check_desc(desc);
    if (rc) return rc;
    if (!keep_dev || !keep_host) return fail(FLEXMOE_EINVAL, "keep_dev / keep_host is NULL");
    KeepArgs args;
    for (int e = 0; e < desc->E; ++e) {
        if (keep_host[e] < 0 || keep_host[e] > desc->I)
            return fail(FLEXMOE_EKEEP, "keep[%d] = %d outside [0, I = %d]", e, keep_host[e], desc->I);
        args.v[e] = keep_host[e];
    }
    for (int e = desc->E; e < kMaxExperts; ++e) args.v[e] = 0;
    set_keep_kernel<<<1, kMaxExperts, 0, (hipStream_t)stream>>>(keep_dev, args, desc->E);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return hip_fail(err, "set_budget launch");
    return FLEXMOE_OK;
}

int flexmoe_rank_reorder(const flexmoe_layer_desc* desc, const float* scores, const void* w_gate,
                         const void* w_up, const void* w_down, void* w_gate_r, void* w_up_r,
                         void* w_down_r, int32_t* perm, void* stream) {
    int rc = check_desc(desc);
    if (rc) return rc;
    if (!scores || !w_gate || !w_up || !w_down || !w_gate_r || !w_up_r || !w_down_r || !perm)
        return fail(FLEXMOE_EINVAL, "rank_reorder: a pointer is NULL");
    const int es = desc->dtype == FLEXMOE_BF16 ? 2 : 4;
    const hipError_t err = launch_rank_reorder(scores, w_gate, w_up, w_down, w_gate_r, w_up_r,
                                               w_down_r, perm, desc->E, desc->I, desc->d, es,
                                               (hipStream_t)stream);
    if (err != hipSuccess) return hip_fail(err, "rank_reorder launch");
    return FLEXMOE_OK;
}

}  // extern "C"

namespace {

// The forward of both weight layouts.  clipped = 0: ranked weights (online
// clipping, any keep table); clipped = 1: the packed weights of one exported
// budget, holding packed_limit channels per matrix.
// The bucketed forward (the paper's Alg. 2 as an ablation of the ragged
// design): routed experts are grouped by retained width k_e, each group's
// GEMMs run as their own launch pair and compute AlignUp(k_e, k_align)
// channels (capped at I), whose extra activations are zeroed.
struct BucketPlan {
    std::vector<int> order;   // expert ids, grouped by width (widest first), id ascending inside
    std::vector<int> kg;      // GEMM width of each expert
    std::vector<int> start;   // first position in `order` of each group, plus the end
    std::vector<int> width;   // the group's aligned width
};

BucketPlan make_plan(const int32_t* keep, int E, int I, int k_align) {
    BucketPlan b;
    std::vector<int> ids(E);
    for (int e = 0; e < E; ++e) ids[e] = e;
    std::stable_sort(ids.begin(), ids.end(), [&](int a, int c) { return keep[a] > keep[c]; });
    b.kg.assign(E, 0);
    for (int i = 0; i < E; ++i) {
        const int e = ids[i], k = keep[e];
        b.order.push_back(e);
        if (k <= 0) continue;  // inactive experts come last and form no group
        b.kg[e] = std::min(I, (k + k_align - 1) / k_align * k_align);
        if (i == 0 || keep[ids[i - 1]] != k) {
            b.start.push_back(i);
            b.width.push_back(b.kg[e]);
        }
    }
    int end = 0;
    while (end < E && keep[b.order[end]] > 0) ++end;
    b.start.push_back(end);
    return b;
}

// What the training forwards keep besides the output (TrainKeep::mode):
//   1: g, u of the routed rows (fragment-blocked) and their h transposed
//      (channel saliency); the combine writes dY = y - target in fp32
//      instead of y;
//   2: g and u of every row, fragment-blocked (the masked layer's backward);
//      the gate/up GEMM computes all I channels of every active expert, the
//      down GEMM only the kept ones.
// Both always run the prefill tile kernels and an unsplit shared down GEMM
// (one shared row set), so the workspace regions after the forward's are
// those of layout(D, T, T).
struct TrainKeep {
    int mode;
    bf16_t *G, *U, *Gs, *Us;  // fragment-blocked g, u
    bf16_t* ht;               // mode 1: transposed h
    int ldt;
    const float* y_target;    // mode 1
    float* dy;
};

int forward_impl(const flexmoe_layer_desc* desc, int32_t T, const void* x, const float* logits,
                 const void* w_gate_r, const void* w_up_r, const void* w_down_r, const int32_t* keep_dev,
                 int clipped, int packed_limit, const int32_t* bucket_keep, int k_align,
                 const void* ws_gate, const void* ws_up, const void* ws_down, void* y, void* workspace,
                 size_t workspace_bytes, const flexmoe_route_out* dbg, void* stream,
                 const TrainKeep* tr = nullptr, bool allow_side = true) {
    int rc = check_desc(desc);
    if (rc) return rc;
    const flexmoe_layer_desc& D = *desc;
    const int train = tr ? tr->mode : 0;
    const bool bucketed = bucket_keep != nullptr;
    if (bucketed) {
        if (k_align < 1) return fail(FLEXMOE_EINVAL, "k_align = %d must be positive", k_align);
        for (int e = 0; e < D.E; ++e)
            if (bucket_keep[e] < 0 || bucket_keep[e] > D.I)
                return fail(FLEXMOE_EKEEP, "keep[%d] = %d outside [0, I = %d]", e, bucket_keep[e], D.I);
    }
    if (T < 0) return fail(FLEXMOE_EINVAL, "T = %d is negative", T);
    if (T > D.max_tokens) return fail(FLEXMOE_ESHAPE, "T = %d exceeds max_tokens = %d", T, D.max_tokens);
    if (T == 0) return FLEXMOE_OK;
    if (!x || !logits || !w_gate_r || !w_up_r || !w_down_r || (!keep_dev && !bucketed) || (!y && train != 1))
        return fail(FLEXMOE_EINVAL, "forward: an input/output pointer is NULL");
    for (const void* ptr : {x, w_gate_r, w_up_r, w_down_r, ws_gate, ws_up, ws_down, (const void*)y})
        if (((uintptr_t)ptr) & 15) return fail(FLEXMOE_EINVAL, "x, weights and y must be 16-byte aligned");
    if (((uintptr_t)logits) & 3 || (!bucketed && ((uintptr_t)keep_dev) & 3))
        return fail(FLEXMOE_EINVAL, "logits and keep_dev must be 4-byte aligned");
    const bool has_shared = D.I_shared > 0;
    if (has_shared != (ws_gate && ws_up && ws_down) || (!has_shared && (ws_gate || ws_up || ws_down)))
        return fail(FLEXMOE_EINVAL, "shared weights must be given iff I_shared > 0");
    const Layout L = layout(D, T, (size_t)T * (train ? 1 : shared_parts(D, T)));
    if (!workspace || workspace_bytes < L.total)
        return fail(FLEXMOE_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes, L.total);
    if (((uintptr_t)workspace) & 255) return fail(FLEXMOE_EWORKSPACE, "workspace is not 256-byte aligned");

    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    int32_t* idx = (int32_t*)(ws + L.idx);
    float* wts = (float*)(ws + L.wts);
    int32_t* blockcnt = (int32_t*)(ws + L.blockcnt);
    int32_t* blockbase = (int32_t*)(ws + L.blockbase);
    int32_t* counts = (int32_t*)(ws + L.counts);
    int32_t* offsets = (int32_t*)(ws + L.offsets);
    int32_t* perm = (int32_t*)(ws + L.perm);
    int32_t* pos = (int32_t*)(ws + L.pos);
    SegMeta* seg = (SegMeta*)(ws + L.seg);
    int32_t* t1 = (int32_t*)(ws + L.t1);
    int32_t* t2 = (int32_t*)(ws + L.t2);
    int32_t* ord2 = (int32_t*)(ws + L.ord2);
    void* O = ws + L.O;
    void* Os = ws + L.Os;
    int32_t* plan = nullptr;
    BucketPlan bp;
    if (bucketed) {
        bp = make_plan(bucket_keep, D.E, D.I, k_align);
        KeepArgs ka, oa, ga;
        for (int e = 0; e < kMaxExperts; ++e) {
            ka.v[e] = e < D.E ? bucket_keep[e] : 0;
            oa.v[e] = e < D.E ? bp.order[e] : 0;
            ga.v[e] = e < D.E ? bp.kg[e] : 0;
        }
        keep_dev = (const int32_t*)(ws + L.keep);
        plan = (int32_t*)(ws + L.plan);
        set_plan_kernel<<<1, kMaxExperts, 0, (hipStream_t)stream>>>((int32_t*)(ws + L.keep), plan, ka, oa, ga,
                                                                     D.E);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "plan upload");
    }
    const int NB = num_chunks(T);
    const int nseg = D.E + (has_shared ? 1 : 0);
    const bool bf16 = D.dtype == FLEXMOE_BF16;
    // kernel family: weight streaming for decode-sized T, large MFMA tiles
    // otherwise (bf16); LDS-tiled FMA for fp32
    const bool decode = bf16 && T <= kDecodeMaxT && !train;
    const int ks2 = train ? 0 : shared_ks2(D, T);
    const int parts = train ? (has_shared ? 1 : 0) : shared_parts(D, T);
    if (train == 2) {
        // every active expert's gate/up GEMM over all I channels, experts in id order
        KeepArgs order, full;
        for (int e = 0; e < kMaxExperts; ++e) {
            order.v[e] = e < D.E ? e : 0;
            full.v[e] = e < D.E ? D.I : 0;
        }
        plan = (int32_t*)(ws + L.plan);
        set_keep_kernel<<<1, kMaxExperts, 0, (hipStream_t)stream>>>(plan, order, D.E);
        set_keep_kernel<<<1, kMaxExperts, 0, (hipStream_t)stream>>>(plan + D.E, full, D.E);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "plan upload");
    }
    // Weight-streaming tiles: up to kGemvMaxT tokens the routed experts run
    // 16-wide tiles on the vector ALUs; above, 64-wide tiles on the matrix
    // cores, whose workgroups share the token rows through LDS (measured on
    // the Qwen2-57B shape: 5-15 % faster per decode step from 9 to 48 tokens
    // than 16-wide matrix-core tiles).  The shared expert (T rows) takes the
    // wide tiles from kDecodeWideSharedT + 1 = 6 tokens on.
    const bool wide_sh = decode && T > kDecodeWideSharedT;
    const bool wide_rt = decode && T > kGemvMaxT;
    const int dbn = wide_rt ? kDecWideBN : kDecBN;
    const TileShape ts = !bf16   ? TileShape{kF32BM, kF32BN, kF32BM, kF32BN, 0}
                         : decode ? TileShape{kDecodeMaxT, dbn, kDecodeMaxT, dbn, ks2}
                                  : TileShape{kBigBM1, kBigBN1, kBigBM2, kBigBN2, ks2};
    // The shared expert's tile width.  On the side stream (every decode-sized
    // batch that may use it) its launches count their own tiles, of the
    // wide shape from kDecodeWideSharedT tokens on; in the launches over all
    // segments its tiles are those the dispatch counts, of the routed shape.
    const bool side_ok = allow_side && has_shared && !train;
    const bool sh_wide_tiles = side_ok && wide_sh;
    const int sbn1 = sh_wide_tiles ? kDecWideBN : ts.bn1, sbn2 = sh_wide_tiles ? kDecWideBN : ts.bn2;

    hipError_t err;
    // grid upper bounds from host-known sizes: the routed part's from the
    // row-tile bound, the shared part's exactly
    const long long rt1 = routed_row_tiles_ub(T, D.E, D.top_k, ts.bm1);
    const long long rt2 = routed_row_tiles_ub(T, D.E, D.top_k, ts.bm2);
    const long long g1r = rt1 * ceil_div(D.I, ts.bn1);
    const long long g2r = rt2 * ceil_div(D.d, ts.bn2);
    const long long g1s = has_shared ? (long long)ceil_div(T, ts.bm1) * ceil_div(D.I_shared, sbn1) : 0;
    const long long g2s = has_shared ? (long long)ceil_div(T, ts.bm2) * ceil_div(D.d, sbn2) * parts : 0;
    if (g1r + g1s > 0x7fffffffLL || g2r + g2s > 0x7fffffffLL) return fail(FLEXMOE_ESHAPE, "tile grid too large");

    // The two GEMMs over one part of the tile list (n1, n2 workgroups), on
    // one stream.
    // the shared expert's GEMMs on the side stream (see below)
    const bool use_side = side_ok && (decode || g1s < (long long)kSideWaves * kComputeUnits);

    auto gemms = [&](int part, int seg_lo, int seg_hi, long long n1, long long n2, hipStream_t st) -> int {
        const bool sh = part == kPartShared;
        const int k1 = sh ? FLEXMOE_K_GATE_UP_SHARED : FLEXMOE_K_GATE_UP;
        const int k2 = sh ? FLEXMOE_K_DOWN_SHARED : FLEXMOE_K_DOWN;
        const bool wide = sh ? wide_sh : wide_rt;
        hipError_t e;
        if (bf16) {
            Gemm1Params<bf16_t> p1{(const bf16_t*)x, (const bf16_t*)w_gate_r, (const bf16_t*)w_up_r,
                                   (const bf16_t*)ws_gate, (const bf16_t*)ws_up, perm, seg, t1,
                                   (bf16_t*)(ws + L.H), (bf16_t*)(ws + L.Hs), D.d, D.I, D.I_shared, D.E,
                                   D.top_k, nseg, T, part, seg_lo, seg_hi, (int)g1s, clipped};
            if (tr) {
                p1.ht = tr->ht;
                p1.ldt = tr->ldt;
                p1.G = tr->G;
                p1.U = tr->U;
                p1.Gs = tr->Gs;
                p1.Us = tr->Us;
            }
            {
                KernelTimer kt(k1, st);
                e = wide         ? launch_gemm1_decode_wide(p1, (int)n1, st)
                    : decode     ? launch_gemm1_decode(p1, (int)n1, st)
                    : train == 1 ? launch_gemm1_big_train(p1, (int)n1, st)
                    : train == 2 ? launch_gemm1_big_train_rm(p1, (int)n1, st)
                                 : launch_gemm1_big(p1, (int)n1, st, !sh, !use_side);
            }
            if (e != hipSuccess) return hip_fail(e, "gate/up GEMM launch");
            // the masked layer's down GEMM reduces over the kept channels only
            if (train == 2 && !sh && (e = launch_seg_use_kept(seg, nseg, st)) != hipSuccess)
                return hip_fail(e, "segment width launch");
            Gemm2Params<bf16_t> p2{(const bf16_t*)(ws + L.H), (const bf16_t*)(ws + L.Hs),
                                   (const bf16_t*)w_down_r, (const bf16_t*)ws_down, seg, t2, (bf16_t*)O,
                                   (bf16_t*)Os, D.d, D.I, D.I_shared, D.E, nseg, T, ks2, part, seg_lo,
                                   seg_hi, (int)g2s, clipped};
            p2.order = ord2;
            {
                KernelTimer kt(k2, st);
                e = wide     ? launch_gemm2_decode_wide(p2, (int)n2, st)
                    : decode ? launch_gemm2_decode(p2, (int)n2, st)
                             : launch_gemm2_big(p2, (int)n2, st, !sh);
            }
            if (e != hipSuccess) return hip_fail(e, "down GEMM launch");
        } else {
            Gemm1Params<float> p1{(const float*)x, (const float*)w_gate_r, (const float*)w_up_r,
                                  (const float*)ws_gate, (const float*)ws_up, perm, seg, t1,
                                  (float*)(ws + L.H), (float*)(ws + L.Hs), D.d, D.I, D.I_shared, D.E,
                                  D.top_k, nseg, T, part, seg_lo, seg_hi, (int)g1s, clipped};
            {
                KernelTimer kt(k1, st);
                e = launch_gemm1_f32(p1, (int)n1, st);
            }
            if (e != hipSuccess) return hip_fail(e, "gate/up GEMM launch");
            Gemm2Params<float> p2{(const float*)(ws + L.H), (const float*)(ws + L.Hs),
                                  (const float*)w_down_r, (const float*)ws_down, seg, t2, (float*)O,
                                  (float*)Os, D.d, D.I, D.I_shared, D.E, nseg, T, 0, part, seg_lo, seg_hi,
                                  (int)g2s, clipped};
            p2.order = ord2;
            {
                KernelTimer kt(k2, st);
                e = launch_gemm2_f32(p2, (int)n2, st);
            }
            if (e != hipSuccess) return hip_fail(e, "down GEMM launch");
        }
        return FLEXMOE_OK;
    };

    // The shared expert's chain runs on the side stream, forked before the
    // routing (it needs none); the routed chain follows the routing on the
    // caller's stream; the combine waits for both.  This pays where the tails
    // of the GEMMs and
    // the routing kernels leave compute units idle: decode-sized batches and
    // shared experts whose gate/up GEMM alone fills fewer than kSideWaves
    // waves of tiles.  Past that, one launch over all segments keeps each
    // XCD's L2 serving one GEMM at a time.
    // The training forwards compute every routed channel (the routed GEMMs
    // alone fill the chip): one launch over all segments there (measured 2 %
    // faster than the split on the Qwen1.5 shape).
    SideStream* side = nullptr;
    std::unique_lock<std::mutex> side_lock;
    if (use_side) {
        if ((rc = side_stream(&side)) != FLEXMOE_OK) return rc;
        side_lock = std::unique_lock<std::mutex>(side->mu);
        if ((err = hipEventRecord(side->fork, s)) != hipSuccess) return hip_fail(err, "fork record");
    }

    // Routing and dispatch on the caller's stream.  The first routing kernel
    // is submitted before the shared expert's GEMMs (it then reaches the
    // compute units first); the rest follow them.
    const bool small = (long long)T * D.top_k <= kSmallAssign;
    const bool pre_routed = small && T > kSmallRouteT;
    if (small && !pre_routed) {
        // one workgroup routes and dispatches everything (timed as routing)
        KernelTimer kt(FLEXMOE_K_ROUTE, s);
        dispatch_small_kernel<<<1, 64 * kSmallWaves, 0, s>>>(logits, T, D.E, D.top_k, D.norm_topk, keep_dev,
                                                             D.I, D.I_shared, D.d, ts, packed_limit, plan, 0,
                                                             idx, wts, counts, perm, pos, offsets, seg, t1,
                                                             t2, ord2);
        err = hipGetLastError();
        if (err != hipSuccess) return hip_fail(err, "dispatch launch");
    } else {
        KernelTimer kt(FLEXMOE_K_ROUTE, s);
        route_kernel<<<NB, 64 * kRouteTokens, 0, s>>>(logits, T, D.E, D.top_k, D.norm_topk, idx, wts,
                                                      blockcnt, NB);
        err = hipGetLastError();
        if (err != hipSuccess) return hip_fail(err, "route launch");
    }

    if (use_side) {
        if ((err = hipStreamWaitEvent(side->stream, side->fork, 0)) != hipSuccess)
            return hip_fail(err, "fork wait");
        if ((rc = gemms(kPartShared, 0, 0, g1s, g2s, side->stream)) != FLEXMOE_OK) return rc;
        if ((err = hipEventRecord(side->join, side->stream)) != hipSuccess) return hip_fail(err, "join record");
    }

    if (pre_routed) {
        // the tokens are routed; one workgroup dispatches them
        KernelTimer kt(FLEXMOE_K_DISPATCH_SCATTER, s);
        dispatch_small_kernel<<<1, 64 * kSmallWaves, 0, s>>>(logits, T, D.E, D.top_k, D.norm_topk, keep_dev,
                                                             D.I, D.I_shared, D.d, ts, packed_limit, plan, 1,
                                                             idx, wts, counts, perm, pos, offsets, seg, t1,
                                                             t2, ord2);
        err = hipGetLastError();
        if (err != hipSuccess) return hip_fail(err, "dispatch launch");
    } else if (!small) {
        {
            KernelTimer kt(FLEXMOE_K_DISPATCH_SCAN, s);
            dispatch_scan_kernel<<<D.E, 256, 0, s>>>(blockcnt, NB, blockbase, counts);
            err = hipGetLastError();
        }
        if (err != hipSuccess) return hip_fail(err, "dispatch scan launch");
        {
            KernelTimer kt(FLEXMOE_K_DISPATCH_SCATTER, s);
            dispatch_scatter_kernel<<<NB, 64, 0, s>>>(idx, keep_dev, counts, blockbase, T, D.E, D.top_k,
                                                      D.I, D.I_shared, D.d, NB, ts, packed_limit, plan,
                                                      perm, pos, offsets, seg, t1, t2, ord2);
            err = hipGetLastError();
        }
        if (err != hipSuccess) return hip_fail(err, "dispatch scatter launch");
    }

    const int hs = has_shared ? 1 : 0;
    if (!bucketed) {
        if (use_side) rc = gemms(kPartRange, hs, nseg, g1r, g2r, s);
        else rc = gemms(kPartRange, 0, nseg, g1r + g1s, g2r + g2s, s);
        if (rc != FLEXMOE_OK) return rc;
    } else {
        if (!use_side && has_shared && (rc = gemms(kPartRange, 0, 1, g1s, g2s, s)) != FLEXMOE_OK) return rc;
        // one launch pair per width group, grids bounded by the group's size
        for (size_t b = 0; b + 1 < bp.start.size(); ++b) {
            const int nb = bp.start[b + 1] - bp.start[b];
            const long long r1 = std::min(routed_row_tiles_ub(T, D.E, D.top_k, ts.bm1), (long long)nb * ceil_div(T, ts.bm1));
            const long long r2 = std::min(routed_row_tiles_ub(T, D.E, D.top_k, ts.bm2), (long long)nb * ceil_div(T, ts.bm2));
            rc = gemms(kPartRange, hs + bp.start[b], hs + bp.start[b + 1], r1 * ceil_div(bp.width[b], ts.bn1),
                       r2 * ceil_div(D.d, ts.bn2), s);
            if (rc != FLEXMOE_OK) return rc;
        }
    }
    if (use_side) {
        if ((err = hipStreamWaitEvent(s, side->join, 0)) != hipSuccess) return hip_fail(err, "join wait");
        side_lock.unlock();
    }
    {
        KernelTimer kt(FLEXMOE_K_COMBINE, s);
        err = train == 1 ? launch_combine_residual((const bf16_t*)O, (const bf16_t*)Os, pos, wts, T, D.top_k, D.d,
                                                   parts, tr->y_target, tr->dy, s)
                         : launch_combine(O, Os, pos, wts, T, D.top_k, D.d, parts, D.dtype, y, s);
    }
    if (err != hipSuccess) return hip_fail(err, "combine launch");

    if (dbg) {
        const size_t A = (size_t)T * D.top_k;
        struct {
            void* dst;
            const void* src;
            size_t bytes;
        } cp[] = {{dbg->topk_idx, idx, A * 4},          {dbg->topk_w, wts, A * 4},
                  {dbg->counts, counts, (size_t)D.E * 4}, {dbg->offsets, offsets, ((size_t)D.E + 1) * 4},
                  {dbg->perm, perm, A * 4},              {dbg->pos, pos, A * 4}};
        for (auto& c : cp) {
            if (!c.dst) continue;
            if ((err = hipMemcpyAsync(c.dst, c.src, c.bytes, hipMemcpyDeviceToDevice, s)) != hipSuccess)
                return hip_fail(err, "debug copy");
        }
    }
    return FLEXMOE_OK;
}

// Packed channels of the clipped layout of keep_host, or a negative error.
long long clipped_channels(const flexmoe_layer_desc* desc, const int32_t* keep_host) {
    int rc = check_desc(desc);
    if (rc) return rc;
    if (!keep_host) return fail(FLEXMOE_EINVAL, "keep_host is NULL");
    long long c = 0;
    for (int e = 0; e < desc->E; ++e) {
        if (keep_host[e] < 0 || keep_host[e] > desc->I)
            return fail(FLEXMOE_EKEEP, "keep[%d] = %d outside [0, I = %d]", e, keep_host[e], desc->I);
        c += packed_width(keep_host[e]);
    }
    return c;
}

}  // namespace

extern "C" {

int flexmoe_layer_forward(const flexmoe_layer_desc* desc, int32_t T, const void* x,
                          const float* logits, const void* w_gate_r, const void* w_up_r,
                          const void* w_down_r, const int32_t* keep_dev, const void* ws_gate,
                          const void* ws_up, const void* ws_down, void* y, void* workspace,
                          size_t workspace_bytes, const flexmoe_route_out* dbg, void* stream) {
    return forward_impl(desc, T, x, logits, w_gate_r, w_up_r, w_down_r, keep_dev, 0, 0x7fffffff, nullptr, 0,
                        ws_gate, ws_up, ws_down, y, workspace, workspace_bytes, dbg, stream);
}

int flexmoe_layer_forward_noalloc(const flexmoe_layer_desc* desc, int32_t T, const void* x,
                                  const float* logits, const void* w_gate_r, const void* w_up_r,
                                  const void* w_down_r, const int32_t* keep_dev, const void* ws_gate,
                                  const void* ws_up, const void* ws_down, void* y,
                                  const flexmoe_route_out* dbg, void* stream) {
    int rc = check_desc(desc);
    if (rc) return rc;
    if (T < 0) return fail(FLEXMOE_EINVAL, "T = %d is negative", T);
    if (T > desc->max_tokens) return fail(FLEXMOE_ESHAPE, "T = %d exceeds max_tokens = %d", T, desc->max_tokens);
    if (T == 0) return FLEXMOE_OK;
    if (!x || !logits || !w_gate_r || !w_up_r || !w_down_r || !keep_dev || !y)
        return fail(FLEXMOE_EINVAL, "forward_noalloc: an input/output pointer is NULL");
    // the regions of flexmoe_layer_forward's workspace for this T (nothing
    // in them needs to start at zero: every kernel writes what it reads)
    const size_t need = layout(*desc, T, (size_t)T * shared_parts(*desc, T)).total;
    if (need > kNoAllocScratchBytes)
        return fail(FLEXMOE_EWORKSPACE,
                    "T = %d needs %zu bytes of scratch; the no-allocation forward's static scratch holds %zu "
                    "(use flexmoe_layer_forward with a workspace)", T, need, kNoAllocScratchBytes);
    void* ws = nullptr;
    if ((rc = scratch_address(&ws)) != FLEXMOE_OK) return rc;
    // every launch on the caller's stream: no side stream, no events
    return forward_impl(desc, T, x, logits, w_gate_r, w_up_r, w_down_r, keep_dev, 0, 0x7fffffff, nullptr, 0,
                        ws_gate, ws_up, ws_down, y, ws, kNoAllocScratchBytes, dbg, stream, nullptr,
                        /*allow_side=*/false);
}

int64_t flexmoe_clipped_channels(const flexmoe_layer_desc* desc, const int32_t* keep_host) {
    return clipped_channels(desc, keep_host);
}

int flexmoe_export_clipped(const flexmoe_layer_desc* desc, const int32_t* keep_host, const void* w_gate_r,
                           const void* w_up_r, const void* w_down_r, void* w_gate_c, void* w_up_c,
                           void* w_down_c, void* stream) {
    const long long c = clipped_channels(desc, keep_host);
    if (c < 0) return (int)c;
    if (!w_gate_r || !w_up_r || !w_down_r || !w_gate_c || !w_up_c || !w_down_c)
        return fail(FLEXMOE_EINVAL, "export_clipped: a weight pointer is NULL");
    for (const void* ptr : {w_gate_r, w_up_r, w_down_r, (const void*)w_gate_c, (const void*)w_up_c,
                            (const void*)w_down_c})
        if (((uintptr_t)ptr) & 15) return fail(FLEXMOE_EINVAL, "weights must be 16-byte aligned");
    if (c == 0) return FLEXMOE_OK;
    KeepArgs k;
    for (int e = 0; e < kMaxExperts; ++e) k.v[e] = e < desc->E ? keep_host[e] : 0;
    const hipError_t err = launch_export_clipped(k, w_gate_r, w_up_r, w_down_r, w_gate_c, w_up_c, w_down_c,
                                                 desc->E, desc->I, desc->d,
                                                 desc->dtype == FLEXMOE_BF16 ? 2 : 4, (hipStream_t)stream);
    if (err != hipSuccess) return hip_fail(err, "export_clipped launch");
    return FLEXMOE_OK;
}

int flexmoe_layer_forward_clipped(const flexmoe_layer_desc* desc, int32_t T, const void* x,
                                  const float* logits, const void* w_gate_c, const void* w_up_c,
                                  const void* w_down_c, const int32_t* keep_dev, int64_t packed_channels,
                                  const void* ws_gate, const void* ws_up, const void* ws_down, void* y,
                                  void* workspace, size_t workspace_bytes, const flexmoe_route_out* dbg,
                                  void* stream) {
    int rc = check_desc(desc);
    if (rc) return rc;
    if (packed_channels < 0 || packed_channels > (long long)desc->E * packed_width(desc->I))
        return fail(FLEXMOE_EINVAL, "packed_channels = %lld outside [0, E * ceil8(I)]", (long long)packed_channels);
    return forward_impl(desc, T, x, logits, w_gate_c, w_up_c, w_down_c, keep_dev, 1, (int)packed_channels,
                        nullptr, 0, ws_gate, ws_up, ws_down, y, workspace, workspace_bytes, dbg, stream);
}

int flexmoe_layer_forward_bucketed(const flexmoe_layer_desc* desc, int32_t T, const void* x,
                                   const float* logits, const void* w_gate_r, const void* w_up_r,
                                   const void* w_down_r, const int32_t* keep_host, int32_t k_align,
                                   const void* ws_gate, const void* ws_up, const void* ws_down, void* y,
                                   void* workspace, size_t workspace_bytes, const flexmoe_route_out* dbg,
                                   void* stream) {
    if (!keep_host) return fail(FLEXMOE_EINVAL, "keep_host is NULL");
    return forward_impl(desc, T, x, logits, w_gate_r, w_up_r, w_down_r, nullptr, 0, 0x7fffffff, keep_host,
                        k_align, ws_gate, ws_up, ws_down, y, workspace, workspace_bytes, dbg, stream);
}

}  // extern "C"

namespace {

// ---- channel saliency -------------------------------------------------------
struct SalLayout {
    Layout f;  // the forward's regions (shared expert unsplit)
    size_t dy, dO, xt, dot, G, U, ht, dgt, dut, wdt, partial, total;
    int ldt, nI, nM;
};

// Row stride of the transposed activation copies: every routed segment takes
// packed_width(rows) <= rows + 7 rows, so A + 7E bounds the padded total.
long long sal_ldt(const flexmoe_layer_desc& D, int T) {
    return ((long long)T * D.top_k + 7LL * D.E + 7) & ~7LL;
}

SalLayout sal_layout(const flexmoe_layer_desc& D, int T) {
    SalLayout S{};
    S.f = layout(D, T, (size_t)T);
    S.ldt = (int)sal_ldt(D, T);
    S.nI = ceil_div(D.I, kSalTile);
    S.nM = ceil_div(D.d, kSalTile);
    const size_t A = (size_t)T * D.top_k, d = D.d, I = D.I, ldt = S.ldt;
    size_t off = S.f.total;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off += align256(bytes);
        return o;
    };
    S.dy = take((size_t)T * d * 4);
    S.dO = take(A * d * 2);
    S.xt = take(d * ldt * 2);
    S.dot = take(d * ldt * 2);
    const size_t A32 = (A + 31) & ~size_t(31);  // fragment-blocked rows
    S.G = take(A32 * I * 2);
    S.U = take(A32 * I * 2);
    S.ht = take(I * ldt * 2);
    S.dgt = take(I * ldt * 2);
    S.dut = take(I * ldt * 2);
    S.wdt = take((size_t)D.E * I * d * 2);
    S.partial = take(3 * (size_t)D.E * I * S.nM * kSalWaveM * 4);
    S.total = off;
    return S;
}

int check_saliency_shape(const flexmoe_layer_desc& D, int T) {
    if (D.dtype != FLEXMOE_BF16) return fail(FLEXMOE_EDTYPE, "channel saliency runs on bf16 layers only");
    if (T < 0) return fail(FLEXMOE_EINVAL, "T = %d is negative", T);
    if (T > D.max_tokens) return fail(FLEXMOE_ESHAPE, "T = %d exceeds max_tokens = %d", T, D.max_tokens);
    if ((long long)std::max(D.d, D.I) * sal_ldt(D, T) >= (1LL << 30))
        return fail(FLEXMOE_ESHAPE, "max(d, I) * (T * top_k + 7 * E) must stay below 2^30");
    return FLEXMOE_OK;
}

int saliency_impl(const flexmoe_layer_desc* desc, int32_t T, const void* x, const float* logits,
                  const void* w_gate, const void* w_up, const void* w_down, const void* w_down_t,
                  const void* ws_gate, const void* ws_up, const void* ws_down, const float* y_target, float scale,
                  float* scores, void* workspace, size_t workspace_bytes, void* stream) {
    int rc = check_desc(desc);
    if (rc) return rc;
    const flexmoe_layer_desc& D = *desc;
    if ((rc = check_saliency_shape(D, T)) != FLEXMOE_OK) return rc;
    if (T == 0) return FLEXMOE_OK;
    if (!x || !logits || !w_gate || !w_up || !w_down || !y_target || !scores)
        return fail(FLEXMOE_EINVAL, "saliency: an input/output pointer is NULL");
    for (const void* ptr : {x, w_gate, w_up, w_down, w_down_t, ws_gate, ws_up, ws_down, (const void*)y_target})
        if (((uintptr_t)ptr) & 15) return fail(FLEXMOE_EINVAL, "x, weights and y_target must be 16-byte aligned");
    if (((uintptr_t)logits) & 3 || ((uintptr_t)scores) & 3)
        return fail(FLEXMOE_EINVAL, "logits and scores must be 4-byte aligned");
    const bool has_shared = D.I_shared > 0;
    if (has_shared != (ws_gate && ws_up && ws_down) || (!has_shared && (ws_gate || ws_up || ws_down)))
        return fail(FLEXMOE_EINVAL, "shared weights must be given iff I_shared > 0");
    const SalLayout S = sal_layout(D, T);
    if (!workspace || workspace_bytes < S.total)
        return fail(FLEXMOE_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes, S.total);
    if (((uintptr_t)workspace) & 255) return fail(FLEXMOE_EWORKSPACE, "workspace is not 256-byte aligned");

    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    const Layout& L = S.f;
    float* wts = (float*)(ws + L.wts);
    int32_t* perm = (int32_t*)(ws + L.perm);
    SegMeta* seg = (SegMeta*)(ws + L.seg);
    int32_t* keep = (int32_t*)(ws + L.keep);
    float* dy = (float*)(ws + S.dy);
    bf16_t* dO = (bf16_t*)(ws + S.dO);
    bf16_t* xt = (bf16_t*)(ws + S.xt);
    bf16_t* dot = (bf16_t*)(ws + S.dot);
    bf16_t* G = (bf16_t*)(ws + S.G);
    bf16_t* U = (bf16_t*)(ws + S.U);
    bf16_t* ht = (bf16_t*)(ws + S.ht);
    bf16_t* dgt = (bf16_t*)(ws + S.dgt);
    bf16_t* dut = (bf16_t*)(ws + S.dut);
    const bf16_t* wdt = w_down_t ? (const bf16_t*)w_down_t : (const bf16_t*)(ws + S.wdt);
    float* partial = (float*)(ws + S.partial);
    const int hs = has_shared ? 1 : 0, nseg = D.E + hs;
    hipError_t err;

    // 1. the transposed down weights, unless the caller made them
    if (!w_down_t) {
        KernelTimer kt(FLEXMOE_K_SAL_TRANSPOSE, s);
        err = launch_transpose_batched((const bf16_t*)w_down, (bf16_t*)(ws + S.wdt), D.E, D.d, D.I, s);
        if (err != hipSuccess) return hip_fail(err, "down-weight transpose launch");
    }

    // 2. the unpruned layer's forward (every k_e = I), keeping transposed g,
    //    u, h of the routed rows, with dY = Y - target from its combine
    KeepArgs ka;
    for (int e = 0; e < kMaxExperts; ++e) ka.v[e] = e < D.E ? D.I : 0;
    set_keep_kernel<<<1, kMaxExperts, 0, s>>>(keep, ka, D.E);
    if ((err = hipGetLastError()) != hipSuccess) return hip_fail(err, "keep upload");
    static_assert(kBigBM1 == kSalTile, "segment row tiles (rt0) are counted in saliency tile rows");
    const TrainKeep tk{1, G, U, nullptr, nullptr, ht, S.ldt, y_target, dy};
    rc = forward_impl(desc, T, x, logits, w_gate, w_up, w_down, keep, 0, 0x7fffffff, nullptr, 0, ws_gate, ws_up,
                      ws_down, nullptr, workspace, workspace_bytes, nullptr, stream, &tk);
    if (rc != FLEXMOE_OK) return rc;
    const long long gd = routed_row_tiles_ub(T, D.E, D.top_k, kSalTile) * S.nI;
    if (gd > 0x7fffffffLL || 3LL * D.E * S.nI * S.nM > 0x7fffffffLL)
        return fail(FLEXMOE_ESHAPE, "tile grid too large");

    // 3. backward: transposed x and dO, dgrad + SwiGLU backward, wgrad + Eq. 2
    {
        SalPrepParams pp{(const bf16_t*)x, dy, perm, wts, seg, xt, dot, dO, D.d, D.top_k, hs, nseg, S.ldt};
        KernelTimer kt(FLEXMOE_K_SAL_PREP, s);
        err = launch_sal_prep(pp, s);
    }
    if (err != hipSuccess) return hip_fail(err, "saliency prep launch");
    {
        ActDgradParams pd{dO, nullptr, wdt, nullptr, G, U, nullptr, nullptr, seg, dgt, dut, nullptr, nullptr,
                          nullptr, hs, nseg, D.d, D.I, D.I_shared, T, S.nI, 1, S.ldt};
        KernelTimer kt(FLEXMOE_K_SAL_DGRAD, s);
        err = launch_sal_dgrad(pd, gd, s);
    }
    if (err != hipSuccess) return hip_fail(err, "dgrad launch");
    {
        SalWgradParams pw{{xt, xt, dot}, {dgt, dut, ht}, {(const bf16_t*)w_gate, (const bf16_t*)w_up, wdt},
                          seg, partial, hs, D.d, D.I, D.E, S.ldt, S.nI, S.nM};
        KernelTimer kt(FLEXMOE_K_SAL_WGRAD, s);
        err = launch_sal_wgrad(pw, s);
    }
    if (err != hipSuccess) return hip_fail(err, "wgrad launch");
    {
        KernelTimer kt(FLEXMOE_K_SAL_REDUCE, s);
        err = launch_sal_reduce(partial, D.E, D.I, S.nM * kSalWaveM, scale, scores, s);
    }
    if (err != hipSuccess) return hip_fail(err, "saliency reduce launch");
    return FLEXMOE_OK;
}

}  // namespace

extern "C" {

size_t flexmoe_saliency_workspace_bytes(const flexmoe_layer_desc* desc, int32_t T) {
    if (check_desc(desc) != FLEXMOE_OK) return 0;
    if (check_saliency_shape(*desc, T) != FLEXMOE_OK) return 0;
    return sal_layout(*desc, T).total;
}

int flexmoe_channel_saliency(const flexmoe_layer_desc* desc, int32_t T, const void* x, const float* logits,
                             const void* w_gate, const void* w_up, const void* w_down, const void* w_down_t,
                             const void* ws_gate, const void* ws_up, const void* ws_down, const float* y_target,
                             float scale, float* scores, void* workspace, size_t workspace_bytes, void* stream) {
    return saliency_impl(desc, T, x, logits, w_gate, w_up, w_down, w_down_t, ws_gate, ws_up, ws_down, y_target,
                         scale, scores, workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace {

// ---- action learning: training step of the masked layer --------------------
struct TrainLayout {
    Layout f;  // the forward's regions (shared expert unsplit)
    size_t G, U, Gs, Us, dO, dYs, dG, dU, dGs, dUs, dXr, dXs, dmp, stat, total;
    long long rt;  // bound on the routed row tiles
};

TrainLayout train_layout(const flexmoe_layer_desc& D, int T) {
    TrainLayout S{};
    S.f = layout(D, T, (size_t)T);
    S.rt = routed_row_tiles_ub(T, D.E, D.top_k, kTrainTile);
    const size_t A = (size_t)T * D.top_k, d = D.d, I = D.I, Is = D.I_shared, Tz = T;
    size_t off = S.f.total;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off += align256(bytes);
        return o;
    };
    const size_t A32 = (A + 31) & ~size_t(31), T32 = (Tz + 31) & ~size_t(31);  // fragment-blocked rows
    S.G = take(A32 * I * 2);
    S.U = take(A32 * I * 2);
    S.Gs = take(T32 * Is * 2);
    S.Us = take(T32 * Is * 2);
    S.dO = take(A * d * 2);
    S.dYs = take(Tz * d * 2);
    S.dG = take(A * I * 2);
    S.dU = take(A * I * 2);
    S.dGs = take(Tz * Is * 2);
    S.dUs = take(Tz * Is * 2);
    S.dXr = take(A * d * 4);
    S.dXs = take(Tz * d * 4);
    S.dmp = take((size_t)S.rt * kTrainWaveM * I * 4);
    S.stat = take((size_t)D.E * 2 * 4);
    S.total = off;
    return S;
}

int check_train(const flexmoe_layer_desc* desc, int T) {
    int rc = check_desc(desc);
    if (rc) return rc;
    if (desc->dtype != FLEXMOE_BF16) return fail(FLEXMOE_EDTYPE, "action learning runs on bf16 layers only");
    if (T < 0) return fail(FLEXMOE_EINVAL, "T = %d is negative", T);
    if (T > desc->max_tokens) return fail(FLEXMOE_ESHAPE, "T = %d exceeds max_tokens = %d", T, desc->max_tokens);
    return FLEXMOE_OK;
}

int action_widths(const flexmoe_layer_desc& D, const flexmoe_action_set* a, ActionWidths& aw) {
    if (!a) return fail(FLEXMOE_EINVAL, "actions is NULL");
    if (a->K < 1 || a->K > FLEXMOE_MAX_ACTIONS)
        return fail(FLEXMOE_EINVAL, "K = %d actions outside [1, %d]", a->K, FLEXMOE_MAX_ACTIONS);
    aw = ActionWidths{};
    aw.K = a->K;
    for (int k = 0; k < a->K; ++k) {
        const double r = a->ratio[k];
        if (!(r > 0.0 && r <= 1.0)) return fail(FLEXMOE_EINVAL, "ratio[%d] = %g outside (0, 1]", k, r);
        aw.ratio[k] = (float)a->ratio[k];
        aw.width[k] = std::max(1, flexmoe_keep_from_ratio(r, D.I));
    }
    return FLEXMOE_OK;
}

// The regions of the training workspace the backward reads or writes (the
// forward's own regions are carved by forward_impl).
struct TrainPtrs {
    int32_t *idx, *offsets, *perm, *pos;
    float* wts;
    SegMeta* seg;
    bf16_t *O, *G, *U, *Gs, *Us, *dO, *dYs, *dG, *dU, *dGs, *dUs;
    float *dXr, *dXs, *dmp;
};

TrainPtrs train_ptrs(const TrainLayout& S, void* workspace) {
    char* ws = (char*)workspace;
    const Layout& L = S.f;
    TrainPtrs P;
    P.idx = (int32_t*)(ws + L.idx);
    P.wts = (float*)(ws + L.wts);
    P.offsets = (int32_t*)(ws + L.offsets);
    P.perm = (int32_t*)(ws + L.perm);
    P.pos = (int32_t*)(ws + L.pos);
    P.seg = (SegMeta*)(ws + L.seg);
    P.O = (bf16_t*)(ws + L.O);
    P.G = (bf16_t*)(ws + S.G);
    P.U = (bf16_t*)(ws + S.U);
    P.Gs = (bf16_t*)(ws + S.Gs);
    P.Us = (bf16_t*)(ws + S.Us);
    P.dO = (bf16_t*)(ws + S.dO);
    P.dYs = (bf16_t*)(ws + S.dYs);
    P.dG = (bf16_t*)(ws + S.dG);
    P.dU = (bf16_t*)(ws + S.dU);
    P.dGs = (bf16_t*)(ws + S.dGs);
    P.dUs = (bf16_t*)(ws + S.dUs);
    P.dXr = (float*)(ws + S.dXr);
    P.dXs = (float*)(ws + S.dXs);
    P.dmp = (float*)(ws + S.dmp);
    return P;
}

int check_workspace(const TrainLayout& S, const void* workspace, size_t bytes) {
    if (!workspace || bytes < S.total)
        return fail(FLEXMOE_EWORKSPACE, "workspace of %zu bytes given, %zu needed", bytes, S.total);
    if (((uintptr_t)workspace) & 255) return fail(FLEXMOE_EWORKSPACE, "workspace is not 256-byte aligned");
    return FLEXMOE_OK;
}

}  // namespace

extern "C" {

int flexmoe_transpose_weights(const flexmoe_layer_desc* desc, const void* w_gate, const void* w_up,
                              const void* w_down, const void* ws_gate, const void* ws_up, const void* ws_down,
                              void* w_gate_t, void* w_up_t, void* w_down_t, void* ws_gate_t, void* ws_up_t,
                              void* ws_down_t, void* stream) {
    int rc = check_train(desc, 0);
    if (rc) return rc;
    const flexmoe_layer_desc& D = *desc;
    const void* pairs[6][2] = {{w_gate, w_gate_t}, {w_up, w_up_t},   {w_down, w_down_t},
                               {ws_gate, ws_gate_t}, {ws_up, ws_up_t}, {ws_down, ws_down_t}};
    for (int i = 0; i < 6; ++i) {
        if ((pairs[i][0] == nullptr) != (pairs[i][1] == nullptr))
            return fail(FLEXMOE_EINVAL, "transpose_weights: a weight and its copy must be given together");
        if (i >= 3 && pairs[i][0] && D.I_shared == 0)
            return fail(FLEXMOE_EINVAL, "transpose_weights: shared weights given but I_shared = 0");
    }
    for (const void* ptr : {w_gate, w_up, w_down, ws_gate, ws_up, ws_down, (const void*)w_gate_t,
                            (const void*)w_up_t, (const void*)w_down_t, (const void*)ws_gate_t,
                            (const void*)ws_up_t, (const void*)ws_down_t})
        if (((uintptr_t)ptr) & 15) return fail(FLEXMOE_EINVAL, "weights must be 16-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    hipError_t err;
    struct {
        const void* src;
        void* dst;
        int batch, rows, cols;
    } jobs[] = {{w_gate, w_gate_t, D.E, D.I, D.d},        {w_up, w_up_t, D.E, D.I, D.d},
                {w_down, w_down_t, D.E, D.d, D.I},        {ws_gate, ws_gate_t, 1, D.I_shared, D.d},
                {ws_up, ws_up_t, 1, D.I_shared, D.d},     {ws_down, ws_down_t, 1, D.d, D.I_shared}};
    for (auto& j : jobs) {
        if (!j.src) continue;
        if ((err = launch_transpose_batched((const bf16_t*)j.src, (bf16_t*)j.dst, j.batch, j.rows, j.cols, s)) !=
            hipSuccess)
            return hip_fail(err, "weight transpose launch");
    }
    return FLEXMOE_OK;
}

int flexmoe_sample_actions(const flexmoe_layer_desc* desc, const flexmoe_action_set* actions, const float* alpha,
                           const float* gumbel, int32_t* keep_dev, int32_t* action_dev, void* stream) {
    int rc = check_train(desc, 0);
    if (rc) return rc;
    ActionWidths aw;
    if ((rc = action_widths(*desc, actions, aw)) != FLEXMOE_OK) return rc;
    if (!alpha || !gumbel || !keep_dev) return fail(FLEXMOE_EINVAL, "sample_actions: a pointer is NULL");
    KernelTimer kt(FLEXMOE_K_ACT_OTHER, (hipStream_t)stream);
    const hipError_t err = launch_sample_actions(aw, alpha, gumbel, desc->E, keep_dev, action_dev,
                                                 (hipStream_t)stream);
    if (err != hipSuccess) return hip_fail(err, "sample_actions launch");
    return FLEXMOE_OK;
}

size_t flexmoe_train_workspace_bytes(const flexmoe_layer_desc* desc, int32_t T) {
    if (check_train(desc, T) != FLEXMOE_OK) return 0;
    return train_layout(*desc, T).total;
}

int flexmoe_train_forward(const flexmoe_layer_desc* desc, int32_t T, const void* x, const float* logits,
                          const void* w_gate, const void* w_up, const void* w_down, const int32_t* keep_dev,
                          const void* ws_gate, const void* ws_up, const void* ws_down, void* y, void* workspace,
                          size_t workspace_bytes, void* stream) {
    int rc = check_train(desc, T);
    if (rc) return rc;
    const flexmoe_layer_desc& D = *desc;
    if (T == 0) return FLEXMOE_OK;
    if (!x || !logits || !w_gate || !w_up || !w_down || !keep_dev || !y)
        return fail(FLEXMOE_EINVAL, "train_forward: an input/output pointer is NULL");
    for (const void* ptr : {x, w_gate, w_up, w_down, ws_gate, ws_up, ws_down, (const void*)y})
        if (((uintptr_t)ptr) & 15) return fail(FLEXMOE_EINVAL, "x, weights and y must be 16-byte aligned");
    if (((uintptr_t)logits) & 3 || ((uintptr_t)keep_dev) & 3)
        return fail(FLEXMOE_EINVAL, "logits and keep_dev must be 4-byte aligned");
    const bool has_shared = D.I_shared > 0;
    if (has_shared != (ws_gate && ws_up && ws_down) || (!has_shared && (ws_gate || ws_up || ws_down)))
        return fail(FLEXMOE_EINVAL, "shared weights must be given iff I_shared > 0");
    const TrainLayout S = train_layout(D, T);
    if ((rc = check_workspace(S, workspace, workspace_bytes)) != FLEXMOE_OK) return rc;
    TrainPtrs P = train_ptrs(S, workspace);
    static_assert(kBigBM1 == kTrainTile, "segment row tiles (rt0) are counted in training tile rows");
    const TrainKeep tk{2, P.G, P.U, P.Gs, P.Us, nullptr, 0, nullptr, nullptr};
    return forward_impl(desc, T, x, logits, w_gate, w_up, w_down, keep_dev, 0, 0x7fffffff, nullptr, 0, ws_gate,
                        ws_up, ws_down, y, workspace, workspace_bytes, nullptr, stream, &tk);
}

int flexmoe_train_backward(const flexmoe_layer_desc* desc, int32_t T, const float* logits, const float* dy,
                           const void* w_gate_t, const void* w_up_t, const void* w_down_t, const void* ws_gate_t,
                           const void* ws_up_t, const void* ws_down_t, float* dx, float* dlogits, float* dmask,
                           void* workspace, size_t workspace_bytes, void* stream) {
    int rc = check_train(desc, T);
    if (rc) return rc;
    const flexmoe_layer_desc& D = *desc;
    if (T == 0) return FLEXMOE_OK;
    if (!logits || !dy || !w_gate_t || !w_up_t || !w_down_t || !dx || !dlogits || !dmask)
        return fail(FLEXMOE_EINVAL, "train_backward: an input/output pointer is NULL");
    for (const void* ptr : {(const void*)dy, w_gate_t, w_up_t, w_down_t, ws_gate_t, ws_up_t, ws_down_t,
                            (const void*)dx})
        if (((uintptr_t)ptr) & 15) return fail(FLEXMOE_EINVAL, "dy, dx and weights must be 16-byte aligned");
    if (((uintptr_t)logits) & 3 || ((uintptr_t)dlogits) & 3 || ((uintptr_t)dmask) & 3)
        return fail(FLEXMOE_EINVAL, "logits, dlogits and dmask must be 4-byte aligned");
    const bool has_shared = D.I_shared > 0;
    if (has_shared != (ws_gate_t && ws_up_t && ws_down_t) || (!has_shared && (ws_gate_t || ws_up_t || ws_down_t)))
        return fail(FLEXMOE_EINVAL, "shared weight copies must be given iff I_shared > 0");
    const TrainLayout S = train_layout(D, T);
    if ((rc = check_workspace(S, workspace, workspace_bytes)) != FLEXMOE_OK) return rc;
    TrainPtrs P = train_ptrs(S, workspace);
    hipStream_t s = (hipStream_t)stream;
    hipError_t err;
    const int hs = has_shared ? 1 : 0, nseg = D.E + hs;
    const int A = T * D.top_k;
    const int nI = ceil_div(D.I, kTrainTile), nIs = ceil_div(std::max(D.I_shared, 1), kTrainTile);
    const int nD = ceil_div(D.d, kTrainTile);
    const long long sh_rows = has_shared ? ceil_div(T, kTrainTile) : 0;
    const long long tiles_dgrad = sh_rows * nIs + S.rt * nI;
    const long long tiles_dx = sh_rows * nD + S.rt * nD;
    if (tiles_dgrad > 0x7fffffffLL || tiles_dx > 0x7fffffffLL) return fail(FLEXMOE_ESHAPE, "tile grid too large");
    {
        KernelTimer kt(FLEXMOE_K_ACT_OTHER, s);
        err = launch_train_prep(dy, P.perm, P.wts, P.offsets + D.E, A, T, D.d, D.top_k, P.dO,
                                has_shared ? P.dYs : nullptr, s);
    }
    if (err != hipSuccess) return hip_fail(err, "backward prep launch");
    {
        ActDgradParams pd{P.dO, P.dYs, (const bf16_t*)w_down_t, (const bf16_t*)ws_down_t, P.G, P.U, P.Gs, P.Us,
                          P.seg, P.dG, P.dU, P.dGs, P.dUs, P.dmp, hs, nseg, D.d, D.I, D.I_shared, T, nI, nIs, 0};
        KernelTimer kt(FLEXMOE_K_ACT_DGRAD, s);
        err = launch_act_dgrad(pd, tiles_dgrad, s);
    }
    if (err != hipSuccess) return hip_fail(err, "dgrad launch");
    {
        ActDxParams px{P.dG, P.dU, P.dGs, P.dUs, (const bf16_t*)w_gate_t, (const bf16_t*)w_up_t,
                       (const bf16_t*)ws_gate_t, (const bf16_t*)ws_up_t, P.seg, P.dXr, P.dXs, hs, nseg, D.d, D.I,
                       D.I_shared, T, nD};
        KernelTimer kt(FLEXMOE_K_ACT_DX, s);
        err = launch_act_dx(px, tiles_dx, s);
    }
    if (err != hipSuccess) return hip_fail(err, "dx launch");
    {
        KernelTimer kt(FLEXMOE_K_ACT_OTHER, s);
        err = launch_combine_backward(P.dXr, has_shared ? P.dXs : nullptr, P.O, P.pos, P.idx, P.wts, logits, dy, T,
                                      D.E, D.top_k, D.d, D.norm_topk, dx, dlogits, s);
        if (err == hipSuccess) err = launch_dmask_reduce(P.dmp, P.seg, hs, D.E, D.I, dmask, s);
    }
    if (err != hipSuccess) return hip_fail(err, "combine backward launch");
    return FLEXMOE_OK;
}

int flexmoe_action_grad(const flexmoe_layer_desc* desc, int32_t T, const flexmoe_action_set* actions,
                        const float* alpha, const float* gumbel, float tau, float lambda_cost, float beta,
                        const float* dmask, float* dalpha, float* stats, void* workspace,
                        size_t workspace_bytes, void* stream) {
    int rc = check_train(desc, T);
    if (rc) return rc;
    const flexmoe_layer_desc& D = *desc;
    ActionWidths aw;
    if ((rc = action_widths(D, actions, aw)) != FLEXMOE_OK) return rc;
    if (!(tau > 0.f)) return fail(FLEXMOE_EINVAL, "tau = %g must be positive", (double)tau);
    if (T < 1) return fail(FLEXMOE_EINVAL, "T = %d: the load ratios need at least one token", T);
    if (!alpha || !gumbel || !dmask || !dalpha) return fail(FLEXMOE_EINVAL, "action_grad: a pointer is NULL");
    const TrainLayout S = train_layout(D, T);
    if ((rc = check_workspace(S, workspace, workspace_bytes)) != FLEXMOE_OK) return rc;
    const int32_t* counts = (const int32_t*)((const char*)workspace + S.f.counts);
    float* per_expert = (float*)((char*)workspace + S.stat);
    KernelTimer kt(FLEXMOE_K_ACT_OTHER, (hipStream_t)stream);
    const hipError_t err = launch_action_grad(aw, alpha, gumbel, tau, dmask, counts, (long long)T * D.top_k, D.E,
                                              D.I, lambda_cost, beta, dalpha, per_expert, stats,
                                              (hipStream_t)stream);
    if (err != hipSuccess) return hip_fail(err, "action_grad launch");
    return FLEXMOE_OK;
}

}  // extern "C"
