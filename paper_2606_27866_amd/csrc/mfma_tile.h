// Building blocks of the bf16 MFMA GEMM kernels (gfx950): operands are
// staged in LDS as K tiles of 64 bf16 per row (128-byte rows), loaded straight
// from global memory by buffer_load ... lds, and read back as
// v_mfma_f32_32x32x16_bf16 fragments.
#pragma once

#include "kernels.h"

namespace flexmoe {
namespace mfma {

constexpr int BK = 64;               // K elements per LDS row (one K tile)
constexpr int ROWB = BK * 2;         // bytes per LDS row
constexpr int CHUNKS = ROWB / 16;    // 16-byte chunks per LDS row
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_ptr_t;

// 16 lanes of a fragment read hit 16 consecutive rows at one logical chunk;
// XOR-ing the chunk with row bits 1..3 spreads them over all 64 banks.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & (CHUNKS - 1)); }

// s_waitcnt with vmcnt = n and no wait on expcnt / lgkmcnt (gfx9 encoding).
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitLgkm0 = waitcnt_vm(63) & ~(15 << 8);  // lgkmcnt(0) only

// The 8 K values of `chunk` of LDS row `row` (one lane's MFMA operand).
__device__ __forceinline__ bf16x8 lds_frag(const unsigned char* base, int row, int chunk) {
    return __builtin_bit_cast(bf16x8,
                              *reinterpret_cast<const u32x4*>(base + row * ROWB + swz(row, chunk) * 16));
}

// Raw buffer descriptor over `elems` bf16 elements (the extent must stay
// below 2^31 bytes: the host checks the shapes).  The fourth dword is the
// gfx9 raw-buffer format word.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const bf16_t* base, size_t elems) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(base), (short)0, (int)(elems * 2),
                                             0x00020000);
}
// A byte offset past every descriptor's extent: the load returns zeros (the
// scalar offset added to it stays below 2^31, so it cannot wrap into range).
constexpr uint32_t kOOB = 0x80000000u;

// 16 bytes per lane from base + voff + soff straight into LDS (M0 = lds).
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                           unsigned char* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t*)lds, 16, voff, soff, 0, 0);
}

// A bare s_barrier: a workgroup fence would also drain the DMAs of later K
// tiles that should stay in flight.  Callers wait for their own LDS reads
// and DMAs first.
__device__ __forceinline__ void barrier_no_fence() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Scheduling template for one 16-deep step: NMF MFMAs, NV vector memory
// reads (DMA) and NRD LDS reads, issued round-robin.
template <int NMF, int NV, int NRD>
__device__ __forceinline__ void sched_interleave() {
    constexpr int R = NMF > NRD ? (NMF > NV ? NMF : NV) : (NRD > NV ? NRD : NV);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (r < NMF) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        if (r < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read (DMA)
        if (r < NRD) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
    }
}

}  // namespace mfma
}  // namespace flexmoe
