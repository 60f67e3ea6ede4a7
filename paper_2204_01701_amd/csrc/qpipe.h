// qpipe.h -- the multi-stage global->LDS pipeline shared by the GEMM kernels.
//
// Operand tiles are copied straight from global memory into LDS with
// global_load_lds_dwordx4 (16 bytes per lane, no register staging).  One
// wave-instruction fills 64 consecutive 16-byte LDS slots (1 KiB) starting
// at a wave-uniform base; each lane chooses which 16 global bytes land in
// its slot.  Lanes with nothing to load (padding taps, ragged tile edges)
// read a 16-byte block of zeros instead.
//
// A ring of NS stages is kept in flight.  Iteration s of a K loop:
//   wait until this thread's loads of stage s have landed (vmcnt <= later stages),
//   s_barrier (so every thread's stage-s loads are visible and stage s-1 is consumed),
//   issue the loads of stage s+NS-1 into the slot stage s-1 used,
//   compute stage s.
// The wait and the barrier are one asm statement with a memory clobber, so
// the compiler neither reorders LDS accesses across it nor adds a full
// vmcnt(0) drain (which a __syncthreads() fence would force).
//
// Two LDS tile layouts:
//  * K-contiguous ("KM"): one row per GEMM row, 64 bytes of the reduction
//    index per row per stage (4 slots).  Physical slot = row*4 + (c ^ ((row >> 2) & 3)):
//    the 16-byte MFMA fragment reads of 16 consecutive rows hit 16 distinct bank groups.
//  * natural ("NAT"): one row per reduction index (pixel), the GEMM row index
//    contiguous inside it; read with ds_read_b64_tr_b16, which hands each lane
//    4 consecutive reduction-index values of one GEMM row.  Slots are XOR
//    swizzled so that the four rows one transposed read touches fall in
//    distinct bank groups.
#pragma once

#include "qdevice.h"

namespace ql {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;

// Copy 16 bytes per lane from gptr into LDS at wave_base + 16 * lane.
// Issued as inline asm, so the compiler's wait insertion does not see an LDS
// write in flight: given the builtin, it puts a full vmcnt(0) drain in front
// of every LDS read it cannot tell apart from the DMA target (the transposed
// reads among them), which would leave one step in flight instead of NS - 1.
// Ordering is explicit instead: each ring step waits for its own loads with
// vmcnt and a barrier (below) before any wave reads them, and refills only a
// slot every wave finished reading before the previous barrier.
__device__ __forceinline__ void dma16(const void *gptr, char *wave_base) {
    const uint32_t lds = (uint32_t)reinterpret_cast<uintptr_t>((lds_void_t *)wave_base);
    asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(gptr), "{m0}"(lds));
}

// The same copy through a buffer resource: 16 bytes per lane from byte offset
// voff + soff of the buffer (zeros where voff is at or past its size, so a lane
// with nothing to load passes an out-of-range offset) into LDS at
// wave_base + 16 * lane.  Asm for the same reason as dma16.
__device__ __forceinline__ void dma16_buf(__amdgpu_buffer_rsrc_t rs, uint32_t voff, int soff, char *wave_base) {
    const uint32_t lds = (uint32_t)reinterpret_cast<uintptr_t>((lds_void_t *)wave_base);
    asm volatile("buffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff), "s"(rs), "s"(soff), "{m0}"(lds));
}

// Buffer resource of `bytes` bytes at p (raw: no stride, bounds-checked offsets).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

// The DMA instructions of a K step are numbered 0 .. NI - 1 in issue order;
// a ring may issue them in two parts, issue(step, slot, live, lo, hi) copying
// those numbered lo .. hi - 1.  take() is called once per instruction in
// order (the numbering folds to constants once the issue loops unroll).
struct DmaPart {
    int lo, hi, n;
    __device__ __forceinline__ DmaPart(int l, int h) : lo(l), hi(h), n(0) {}
    __device__ __forceinline__ bool take() {
        const bool t = n >= lo && n < hi;
        ++n;
        return t;
    }
};

// Branch-free choice of a DMA source: the operand address when ok, else the zero page.
__device__ __forceinline__ const void *dma_src(bool ok, const void *p, const void *zero) {
    const uint64_t a = reinterpret_cast<uint64_t>(p), z = reinterpret_cast<uint64_t>(zero);
    return reinterpret_cast<const void *>(ok ? a : z);
}

// Wave index as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Wait until at most N vector-memory operations of this thread are pending,
// then barrier.  gfx9 s_waitcnt: vmcnt in bits [3:0] and [15:14], expcnt and
// lgkmcnt left at their maxima (no wait on them).  The wait goes through the
// builtin, so the compiler's own wait insertion knows what has completed; the
// barrier is asm with a memory clobber, so no LDS access moves across it.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    constexpr int imm = (N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8);
    __builtin_amdgcn_s_waitcnt(imm);
    asm volatile("s_barrier" ::: "memory");
}

// The same, also waiting for this thread's outstanding LDS reads (so a ring
// slot whose fragments every wave has read may be refilled after the barrier).
template <int N>
__device__ __forceinline__ void wait_vm_barrier_lgkm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    constexpr int imm = (N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8);
    __builtin_amdgcn_s_waitcnt(imm);
    asm volatile("s_barrier" ::: "memory");
}

// Plain barrier for LDS hand-offs that involve no DMA (epilogues).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Waits for every outstanding global/DMA operation of this thread.
__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// The software pipeline shared by the GEMM kernels.  A K step is two
// 32-byte chunks; `read(slot, chunk, buf)` loads the MFMA fragments of one
// chunk of the step held in ring slot `slot` into register set `buf` (0/1),
// `mma(buf)` runs the MFMAs on a register set, and `issue(step, slot, live)`
// starts the DMA of a K step into a ring slot (every lane reading the zero
// page when `live` is false).  Step j lives in slot j % NS.
//
// Iteration it (step it; chunk 0 already in register set 0):
//   read chunk 1 of step it into set 1;
//   issue step it + NS - 1 into the slot step it - 1 used, which every wave
//     finished reading before the previous barrier;
//   MFMAs on set 0;
//   wait for step it + 1 and for this wave's LDS reads, barrier;
//   read chunk 0 of step it + 1 into set 0;
//   MFMAs on set 1.
// The compiler interleaves the DMA address arithmetic, the LDS reads and
// the MFMAs within each half.
// Every iteration issues exactly NI DMA instructions per thread (past the
// last step they fill a slot nobody reads again with zeros), so the loop body
// is straight-line code and the vmcnt allowance is the same in every
// iteration.  The last step issues nothing.  NS - 1 steps are in flight
// while a step is being consumed.  With NI1 < NI only the first NI1
// instructions of a step go out before the set-0 MFMAs and the rest after
// the barrier (the wait allowance counts the part already issued).
template <int NS, int NI, int NI1 = NI, class Issue, class Read, class Mma>
__device__ __forceinline__ void run_ring(int nst, int s_begin, Issue &&issue, Read &&read, Mma &&mma) {
    static_assert(NS >= 3 && (NS - 2) * NI < 64 && NI1 >= 1 && NI1 <= NI, "ring depth");
    if (nst <= 0) return;
#pragma unroll
    for (int i = 0; i < NS - 1; ++i) issue(s_begin + i, i, i < nst, 0, NI);
    wait_vm_barrier<(NS - 2) * NI>();
    read(0, 0, 0);
    int slot = 0;
    // The last step is peeled off, so the loop body always takes the barrier
    // path and the compiler's wait before the set-1 MFMAs is not widened by a
    // merge with the barrier-less path.
    for (int it = 0; it < nst - 1; ++it) {
        const int s = s_begin + it + NS - 1, free = slot == 0 ? NS - 1 : slot - 1;
        const bool live = it + NS - 1 < nst;
        read(slot, 1, 1);
        issue(s, free, live, 0, NI1);
        mma(0);
        wait_vm_barrier_lgkm<(NS - 3) * NI + NI1>();
        if constexpr (NI1 < NI) issue(s, free, live, NI1, NI);
        slot = slot + 1 == NS ? 0 : slot + 1;
        read(slot, 0, 0);
        mma(1);
    }
    read(slot, 1, 1);
    mma(0);
    mma(1);
    wait_vm_all();  // the zero-filling DMAs of the last iterations land before the LDS is released
}

// The same pipeline with ONE register set of fragments, for kernels that run
// two waves per SIMD and need the registers for accumulators: each of the CH
// chunks of a step is read and then multiplied; the other wave on the SIMD
// covers the LDS latency.
template <int NS, int NI, int CH = 2, int NI1 = NI, class Issue, class Read, class Mma>
__device__ __forceinline__ void run_ring_single(int nst, int s_begin, Issue &&issue, Read &&read, Mma &&mma) {
    static_assert(NS >= 3 && (NS - 2) * NI < 64 && NI1 >= 1 && NI1 <= NI, "ring depth");
    static_assert(CH >= 2 || NI1 == NI, "the second part goes out after the first half of the chunks");
    if (nst <= 0) return;
#pragma unroll
    for (int i = 0; i < NS - 1; ++i) issue(s_begin + i, i, i < nst, 0, NI);
    wait_vm_barrier<(NS - 2) * NI>();
    int slot = 0;
    for (int it = 0; it < nst - 1; ++it) {
        const int s = s_begin + it + NS - 1, free = slot == 0 ? NS - 1 : slot - 1;
        const bool live = it + NS - 1 < nst;
        issue(s, free, live, 0, NI1);
#pragma unroll
        for (int ch = 0; ch < CH; ++ch) {
            read(slot, ch, 0);
            mma(0);
            if (ch == CH / 2 - 1 && NI1 < NI) issue(s, free, live, NI1, NI);
        }
        wait_vm_barrier_lgkm<(NS - 2) * NI>();
        slot = slot + 1 == NS ? 0 : slot + 1;
    }
#pragma unroll
    for (int ch = 0; ch < CH; ++ch) {
        read(slot, ch, 0);
        mma(0);
    }
    wait_vm_all();
}

// --- KM layout ---------------------------------------------------------------
// Byte offset of logical 16-byte column c (0..3) of row `row` in a KM tile.
__device__ __forceinline__ int km_off(int row, int c) { return row * 64 + ((c ^ ((row >> 2) & 3)) << 4); }

// The logical column a lane fills when a wave-instruction writes rows
// [16j, 16j + 16) of a KM tile (lane l -> slot l): constant per lane.
__device__ __forceinline__ int km_fill_col(int lane) { return (lane & 3) ^ ((lane >> 4) & 3); }

// --- NAT layout (16-bit elements) --------------------------------------------
// Rows hold S16 16-byte slots; the XOR swizzle keeps the 4 consecutive rows
// read by one ds_read_b64_tr_b16 in distinct bank groups.
template <int S16>
__device__ __forceinline__ int nat_swz(int row) {
    if constexpr (S16 >= 16) return (row & 3) << 2;
    else if constexpr (S16 == 8) return ((row >> 1) & 1) << 2;
    else return 0;
}
template <int S16>
__device__ __forceinline__ int nat_off(int row, int slot) {
    return row * (S16 * 16) + ((slot ^ nat_swz<S16>(row)) << 4);
}

// MFMA operand (32 GEMM rows x 16 reduction values, bf16) from a NAT tile whose
// rows are reduction indices: lane l gets GEMM row m0 + l % 32 and reduction
// values k0 + 8 * (l / 32) .. +8, as two ds_read_b64_tr_b16.  Within each
// group of 16 lanes, lane i of a transposed read receives element i % 4 of the
// 8 bytes addressed by lane 4k + i / 4, for k = 0..3; so lane j of the group
// addresses row k0 + 8 * (g / 2) + 4 * h + j / 4, GEMM columns
// m0 + 16 * (g % 2) + 4 * (j % 4) .. +4.
template <int S16>
__device__ __forceinline__ v4u nat_frag_bf16(const char *tile, int k0, int m0, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int col = m0 + 16 * (g & 1) + 4 * (j & 3);  // element column
    const int slot = col >> 3, within = (col & 7) * 2;
    v4u out;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int row = k0 + 8 * (g >> 1) + 4 * h + (j >> 2);
        const char *p = tile + nat_off<S16>(row, slot) + within;
        const v4s_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t *)(p));
        const v2u w = __builtin_bit_cast(v2u, v);
        out[2 * h] = w.x;
        out[2 * h + 1] = w.y;
    }
    return out;
}

}  // namespace ql
