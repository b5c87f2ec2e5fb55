// Key-chunk staging shared by the SnapKV score kernels: a swizzled LDS layout
// for 64-key chunks of K and the direct-to-LDS loads that fill it.
#pragma once

#include "kve_device.h"

namespace kve {

// One key chunk: kChunkKeys rows of D elements.
constexpr int kChunkKeys = 64;

template <typename T, int D>
struct KChunk {
    static constexpr int ES = (int)sizeof(T);
    static constexpr int ROW = D * ES;            // bytes per key row
    static constexpr int BYTES = kChunkKeys * ROW;
    static constexpr int NC16 = ROW / 16;         // 16-byte pieces per row
    static constexpr int NSTEP = D / Mma<T>::KSTEP;
};

template <typename T, int D>
using QFrag = typename Mma<T>::frag[KChunk<T, D>::NSTEP];

// Byte offset of 16-byte piece c of key row r inside a chunk buffer.  The XOR
// swizzle puts the 32 rows one matrix-core operand reads on distinct bank groups.
template <typename T, int D>
__device__ __forceinline__ int chunk_swz(int r, int c) {
    return r * KChunk<T, D>::ROW + ((c ^ (r & (KChunk<T, D>::NC16 - 1))) << 4);
}

// Matrix-core fragment of key row r at element k (a multiple of KPL).
template <typename T, int D>
__device__ __forceinline__ typename Mma<T>::frag chunk_frag(const char* buf, int r, int k) {
    const int byte = k * KChunk<T, D>::ES;
    return Mma<T>::load(buf + chunk_swz<T, D>(r, byte >> 4) + (byte & 15), 0);
}

// One direct-to-LDS load: lane i's 16 bytes at base + voff (bytes) land in LDS
// at lds_dst + 16 i (lds_dst wave-uniform).  Issued as inline assembly so the
// compiler does not track it: compiler-tracked direct-to-LDS loads make it
// wait for every outstanding load before any LDS read, which would drain the
// chunks kept in flight.  Callers wait with explicit vmcnt counts instead;
// loads the compiler does not know of can only make its own waits stricter
// (memory operations complete in order per wave), never too lenient.
__device__ __forceinline__ void lds_dma16(const char* base, unsigned voff, const char* lds_dst) {
    const unsigned m0 = __builtin_amdgcn_readfirstlane(
        (unsigned)(size_t)(const __attribute__((address_space(3))) char*)lds_dst);
    // the LDS base goes in M0; one wait state must separate its write from the
    // direct-to-LDS load that reads it
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(voff), "s"(base), "{m0}"(m0) : "memory");
}

// Issue direct-to-LDS loads of one chunk, split over `nwaves` waves (this wave
// is number `wv` of them).  Each lane fetches the global piece that the
// swizzled layout keeps at its landing position.  Rows at or past `valid` are
// read from row 0 instead (never from outside the segment) so that every wave
// always issues the same number of loads per chunk; callers mask those keys.
template <typename T, int D, int NWAVES>
__device__ __forceinline__ void chunk_stream(char* slot, const char* rows, int valid, int wv, int lane) {
    using C = KChunk<T, D>;
    static_assert(C::BYTES % (NWAVES * 1024) == 0, "chunk must split into whole 1 KiB wave loads");
#pragma unroll
    for (int j = 0; j < C::BYTES / (NWAVES * 1024); ++j) {
        const int dst = (j * NWAVES + wv) * 1024;  // wave-uniform byte offset
        const int o = dst + lane * 16;
        const int r = o / C::ROW;
        const int c = ((o - r * C::ROW) >> 4) ^ (r & (C::NC16 - 1));
        const unsigned off = r < valid ? (unsigned)(r * C::ROW + c * 16) : (unsigned)(c * 16);
        lds_dma16(rows, off, slot + dst);
    }
}

template <typename T, int D, int NWAVES>
constexpr int chunk_loads_per_wave() {
    return KChunk<T, D>::BYTES / (NWAVES * 1024);
}

// s_waitcnt immediate that waits until at most `n` vector-memory operations
// of this wave are outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt and lgkmcnt left unconstrained).
constexpr int vmcnt_imm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(N));
}

// Wait for every outstanding global load of this wave and keep the compiler
// from moving memory accesses across the wait.  Called once the loads a kernel
// issues before its chunk stream (query fragments, statistics) are issued, so
// that the compiler has no load of its own left to wait for inside the loop,
// where such a wait would also drain the chunk loads in flight.
__device__ __forceinline__ void drain_loads() {
    wait_vmcnt<0>();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Workgroup barrier for LDS traffic only.  __syncthreads() also waits for every
// outstanding global load of the wave, which would drain the chunk loads kept
// in flight ahead of the computation; this barrier waits for the wave's own
// LDS operations (lgkmcnt 0, vmcnt unconstrained) and keeps the compiler from
// moving memory accesses across it.  Direct-to-LDS chunk loads are covered by
// the explicit vmcnt waits before the barrier that publishes their slot.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));  // lgkmcnt(0)
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

}  // namespace kve
