// Key-chunk staging for the streaming score kernels: a swizzled LDS layout for
// chunks of key rows, the direct-to-LDS loads that fill it, and the waits and
// barriers that publish a chunk to every wave of a workgroup.
#pragma once

#include "kve_device.h"

namespace kve {

// One chunk: KEYS key rows of D elements of type T.
template <typename T, int D, int KEYS>
struct KChunk {
    static constexpr int ES = (int)sizeof(T);
    static constexpr int ROW = D * ES;            // bytes per key row
    static constexpr int BYTES = KEYS * ROW;
    static constexpr int NC16 = ROW / 16;         // 16-byte pieces per row
    static constexpr int NSTEP = D / Mma<T>::KSTEP;
};

// Byte offset of 16-byte piece c of key row r inside a chunk buffer.  The XOR
// swizzle puts the eight consecutive rows that one LDS read cycle of a
// matrix-core operand touches (same piece) on distinct 16-byte bank groups.
// It changes only the low three bits of the piece index, so pieces c and
// c + 8 of a row stay 128 bytes apart.
template <int ROW>
__device__ __forceinline__ int chunk_swz(int r, int c) {
    static_assert(ROW >= 128, "rows of at least eight 16-byte pieces");
    return r * ROW + ((c ^ (r & 7)) << 4);
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

// Matrix-core fragments of a chunk, read from LDS with per-lane byte offsets
// worked out once per kernel.  Fragment (kb, st) of lane l is key row
// 32 kb + l%32 (counted from the wave's first key row, `base` bytes into the
// chunk) at k-step st.  With bf16 the swizzled offset of each k-step is
// kept in a register, so that a read is one ds_read_b128 whose slot and
// key-block parts are immediate offsets; fp32 chunks (D/2 k-steps) work the
// offset out at each read.
template <typename T, int D, int KEYS>
struct ChunkReader {
    using C = KChunk<T, D, KEYS>;
    using M = Mma<T>;
    static constexpr bool kTable = sizeof(T) == 2;
    // bf16: k-step st reads piece 2 st + (lane / 32); steps st and st + 4 are
    // 128 bytes apart, so four offsets cover all steps
    static constexpr int NOFF = kTable ? (C::NSTEP < 4 ? C::NSTEP : 4) : 1;
    int off[NOFF];
    int lane, base;

    __device__ __forceinline__ void init(int lane_, int base_) {
        lane = lane_;
        base = base_;
        if constexpr (kTable) {
#pragma unroll
            for (int st = 0; st < NOFF; ++st) off[st] = offset(st);
        }
    }
    __device__ __forceinline__ int offset(int st) const {
        const int byte = (st * M::KSTEP + (lane >> 5) * M::KPL) * C::ES;
        return base + chunk_swz<C::ROW>(lane & 31, byte >> 4) + (byte & 15);
    }
    __device__ __forceinline__ typename M::frag get(const char* slot, int kb, int st) const {
        if constexpr (kTable)
            return M::load(slot + kb * 32 * C::ROW + (st / 4) * 128 + off[st % 4], 0);
        else
            return M::load(slot + kb * 32 * C::ROW + offset(st), 0);
    }
};

// Direct-to-LDS loads of whole chunks with the per-lane global offsets worked
// out once per kernel.  Wave `wv` (wave-uniform) of NWAVES issues LPW loads
// per chunk; load j lands at byte (j * NWAVES + wv) * 1024 of the slot.  A
// chunk with fewer than KEYS valid rows reads row 0 in place of the missing
// rows (never outside the segment), so the number of loads per chunk stays
// fixed; callers mask those keys.
template <typename T, int D, int KEYS, int NWAVES>
struct ChunkWriter {
    using C = KChunk<T, D, KEYS>;
    static constexpr int LPW = C::BYTES / (NWAVES * 1024);
    static_assert(C::BYTES % (NWAVES * 1024) == 0, "chunk must split into whole 1 KiB wave loads");
    unsigned goff[LPW];
    int wv;

    __device__ __forceinline__ void init(int wv_uniform, int lane) {
        wv = wv_uniform;
#pragma unroll
        for (int j = 0; j < LPW; ++j) {
            const int o = (j * NWAVES + wv) * 1024 + lane * 16;
            const int r = o / C::ROW;
            const int c = ((o - r * C::ROW) >> 4) ^ (r & 7);  // inverse of chunk_swz
            goff[j] = (unsigned)(r * C::ROW + c * 16);
        }
    }
    // rows: first key row of the chunk (wave-uniform); valid: rows in bounds
    __device__ __forceinline__ void issue(char* slot, const char* rows, int valid) const {
        if (valid >= KEYS) {
#pragma unroll
            for (int j = 0; j < LPW; ++j) lds_dma16(rows, goff[j], slot + (j * NWAVES + wv) * 1024);
        } else {
#pragma unroll
            for (int j = 0; j < LPW; ++j) {
                const int r = (int)(goff[j] / C::ROW);
                lds_dma16(rows, r < valid ? goff[j] : goff[j] - (unsigned)(r * C::ROW),
                          slot + (j * NWAVES + wv) * 1024);
            }
        }
    }
};

// s_waitcnt immediate that waits until at most `n` vector-memory operations
// of this wave are outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt and lgkmcnt left unconstrained).
constexpr int vmcnt_imm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt holds 6 bits");
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(N));
}

// Wait until this wave's loads of the current chunk have landed while the
// loads of `ahead` (0 .. MAXAHEAD) later chunks, LPW loads each, stay in
// flight.
template <int LPW, int MAXAHEAD>
__device__ __forceinline__ void wait_chunk(int ahead) {
    if constexpr (MAXAHEAD > 0) {
        if (ahead >= MAXAHEAD) {
            wait_vmcnt<MAXAHEAD * LPW>();
            return;
        }
        wait_chunk<LPW, MAXAHEAD - 1>(ahead);
    } else {
        wait_vmcnt<0>();
    }
}

// Materialise a loaded value in registers at this point.  The loads a kernel
// issues before its chunk stream (query fragments, statistics) read memory the
// compiler may treat as invariant, so it could otherwise sink them past the
// first chunk loads or re-load them inside the loop; either would put a wait
// for one of its own loads inside the loop, and that wait would also drain the
// chunk loads in flight.  The empty volatile statement takes the value as an
// in-out operand: the compiler waits for the load before it and has to keep
// the result in a register afterwards.
template <typename V>
__device__ __forceinline__ void pin(V& v) {
    asm volatile("" : "+v"(v));
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
