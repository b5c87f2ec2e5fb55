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

// Byte offset of 16-byte piece c of key row r inside a chunk buffer.  A
// matrix-core operand read (ds_read_b128) serves sixteen lanes, i.e. sixteen
// consecutive rows at the same piece, per LDS cycle; the XOR swizzle of the
// piece index puts them on sixteen distinct 16-byte bank groups.  Rows of
// sixteen or more pieces: piece ^ (r % 16).  Rows of eight pieces (two rows per
// 256-byte bank cycle): piece ^ ((r / 2) % 8).  Rows r and r + 32 share the
// swizzle, so a second 32-row block is an immediate offset away.
template <int ROW>
__device__ __forceinline__ int chunk_swz_bits(int r) {
    static_assert(ROW >= 128, "rows of at least eight 16-byte pieces");
    return ROW >= 256 ? (r & 15) : ((r >> 1) & 7);
}
template <int ROW>
__device__ __forceinline__ int chunk_swz(int r, int c) {
    return r * ROW + ((c ^ chunk_swz_bits<ROW>(r)) << 4);
}

// One direct-to-LDS load: lane i's 16 bytes at base + voff (bytes) land in LDS
// at lds_dst + 16 i (lds_dst wave-uniform).  Issued as inline assembly so the
// compiler does not track it: compiler-tracked direct-to-LDS loads make it
// wait for every outstanding load before any LDS read, which would drain the
// chunks kept in flight.  Callers wait with explicit vmcnt counts instead;
// loads the compiler does not know of can only make its own waits stricter
// (memory operations complete in order per wave), never too lenient.
//
// NT marks the load non-temporal: for data read once (streamed keys), so that
// its lines are the first the caches give up.
template <bool NT = false>
__device__ __forceinline__ void lds_dma16(const char* base, unsigned voff, const char* lds_dst) {
    const unsigned m0 = __builtin_amdgcn_readfirstlane(
        (unsigned)(size_t)(const __attribute__((address_space(3))) char*)lds_dst);
    // the LDS base goes in M0; one wait state must separate its write from the
    // direct-to-LDS load that reads it
    if constexpr (NT)
        asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt"
                     :: "v"(voff), "s"(base), "{m0}"(m0) : "memory");
    else
        asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                     :: "v"(voff), "s"(base), "{m0}"(m0) : "memory");
}

// Matrix-core fragments of a chunk, read from LDS with per-lane byte offsets
// worked out once per kernel.  Fragment (kb, st) of lane l is key row
// 32 kb + l%32 (counted from the wave's first key row, `base` bytes into the
// chunk) at k-step st.  With bf16 the swizzled offset of each k-step is
// kept in a register (k-step st reads piece 2 st + lane / 32), so that a read
// is one ds_read_b128 whose slot and key-block parts are immediate offsets;
// fp32 chunks (D/2 k-steps) work the offset out at each read.
template <typename T, int D, int KEYS>
struct ChunkReader {
    using C = KChunk<T, D, KEYS>;
    using M = Mma<T>;
    static constexpr bool kTable = sizeof(T) == 2;
    static constexpr int NOFF = kTable ? C::NSTEP : 1;
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
            return M::load(slot + kb * 32 * C::ROW + off[st], 0);
        else
            return M::load(slot + kb * 32 * C::ROW + offset(st), 0);
    }
};

// Direct-to-LDS loads of whole chunks with the per-lane global offsets worked
// out once per kernel.  Wave `wv` (wave-uniform) of NWAVES issues LPW loads
// per chunk; load j lands at byte (j * NWAVES + wv) * 1024 of the slot.  Key
// row r of a chunk starts r * row_stride bytes after the chunk's first row (a
// multiple of 16, ROW for dense rows), so rows of a strided view (e.g. a
// token-major cache) load the same way.  A chunk with fewer than KEYS valid
// rows reads row 0 in place of the missing rows (never outside the segment),
// so the number of loads per chunk stays fixed; callers mask those keys.
// NT: non-temporal loads (see lds_dma16).
template <typename T, int D, int KEYS, int NWAVES, bool NT = false>
struct ChunkWriter {
    using C = KChunk<T, D, KEYS>;
    static constexpr int LPW = C::BYTES / (NWAVES * 1024);
    static_assert(C::BYTES % (NWAVES * 1024) == 0, "chunk must split into whole 1 KiB wave loads");
    // chunk rows between a lane's consecutive loads; when they span whole
    // swizzle periods (16 rows) all loads of a lane share its column, so one
    // offset serves them all and the wave-uniform base steps by RJ rows
    static constexpr int RJ = NWAVES * 1024 / C::ROW;
    static constexpr bool kOneOff = RJ % 16 == 0;
    unsigned goff[kOneOff ? 1 : LPW];
    unsigned rstride;
    int wv, lane;

    __device__ __forceinline__ void init(int wv_uniform, int lane_, unsigned row_stride = C::ROW) {
        wv = wv_uniform;
        lane = lane_;
        rstride = row_stride;
#pragma unroll
        for (int j = 0; j < (kOneOff ? 1 : LPW); ++j) {
            const int r = row_of(j);
            const int o = (j * NWAVES + wv) * 1024 + lane * 16;
            const int c = ((o - r * C::ROW) >> 4) ^ chunk_swz_bits<C::ROW>(r);  // inverse of chunk_swz
            goff[j] = (unsigned)r * row_stride + (unsigned)(c * 16);
        }
    }
    // chunk row of this lane's load j
    __device__ __forceinline__ int row_of(int j) const { return ((j * NWAVES + wv) * 1024 + lane * 16) / C::ROW; }
    // byte offset of this lane's load j from the chunk's first row
    __device__ __forceinline__ unsigned off_of(int j) const {
        return kOneOff ? goff[0] + (unsigned)(j * RJ) * rstride : goff[j];
    }
    // rows: first key row of the chunk (wave-uniform); valid: rows in bounds
    __device__ __forceinline__ void issue(char* slot, const char* rows, int valid) const {
        if (valid >= KEYS) {
#pragma unroll
            for (int j = 0; j < LPW; ++j) {
                if constexpr (kOneOff)
                    lds_dma16<NT>(rows + (size_t)(j * RJ) * rstride, goff[0], slot + (j * NWAVES + wv) * 1024);
                else
                    lds_dma16<NT>(rows, goff[j], slot + (j * NWAVES + wv) * 1024);
            }
        } else {
#pragma unroll
            for (int j = 0; j < LPW; ++j) {
                const int r = row_of(j);
                const unsigned o = off_of(j);
                lds_dma16<NT>(rows, r < valid ? o : o - (unsigned)r * rstride, slot + (j * NWAVES + wv) * 1024);
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


// ---------------------------------------------------------------------------
// A ring of RING chunk slots in LDS, filled RING - 1 chunks ahead by all
// NWAVES waves of a workgroup.  The caller names each chunk's first row and
// its number of valid rows with src(c, &rows, &valid).
// ---------------------------------------------------------------------------
template <typename T, int D, int KEYS, int NWAVES, int RING, bool NT = false>
struct ChunkRing {
    using C = KChunk<T, D, KEYS>;
    using Wr = ChunkWriter<T, D, KEYS, NWAVES, NT>;
    Wr wr;
    int nch;

    __device__ __forceinline__ void open(int nchunks, int wave_uniform, int lane, unsigned row_stride = C::ROW) {
        wr.init(wave_uniform, lane, row_stride);
        nch = nchunks;
    }
    template <typename Src>
    __device__ __forceinline__ void issue(char* ring, int c, int slot, const Src& src) const {
        const char* rows;
        int valid;
        src(c, &rows, &valid);
        wr.issue(ring + slot * C::BYTES, rows, valid);
    }
    template <typename Src>
    __device__ __forceinline__ void prologue(char* ring, const Src& src) const {
        for (int c = 0; c < min(RING - 1, nch); ++c) issue(ring, c, c, src);
    }
    // Before step s (slot u = s % RING): wait for this wave's loads of chunk
    // s, publish it with the barrier, then refill the slot of chunk s - 1
    // (read by every wave before the barrier) with chunk s + RING - 1.
    template <typename Src>
    __device__ __forceinline__ void advance(char* ring, int s, int u, const Src& src) const {
        wait_chunk<Wr::LPW, RING - 2>(min(RING - 2, nch - 1 - s));
        lds_barrier();
        if (s + RING - 1 < nch) issue(ring, s + RING - 1, (u + RING - 1) % RING, src);
    }
};

// Products of one chunk's first 64 rows (two 32-row blocks b, fragments from
// LDS) with 32 rows held in registers (reg[st]).  LDS_A: the chunk rows are the
// A operand (element i of acc[b] belongs to chunk row 32 b + c_row(i, lane),
// the lane to register row lane % 32); otherwise the register rows are
// (element i belongs to register row c_row(i, lane) in both blocks, the lane
// to chunk row 32 b + lane % 32).  acc[b] starts at zero or, given `init`, at
// the init value of the A-operand row of each element: init[32 b + c_row(i)]
// with LDS_A, init[c_row(i)] otherwise (rows c_row(4 a .. 4 a + 3) are four
// consecutive floats).
//
// c_init, when given, replaces `init`: acc[b] starts at c_init[LDS_A ? b : 0]
// (values already in registers).
template <typename T, int D, int KEYS, bool LDS_A>
__device__ __forceinline__ void chunk_mma(f32x16 (&acc)[2], const ChunkReader<T, D, KEYS>& rd, const char* slot,
                                          const typename Mma<T>::frag (&reg)[KChunk<T, D, KEYS>::NSTEP],
                                          const float* init, int lane, const f32x16* c_init = nullptr) {
    using M = Mma<T>;
    constexpr int NS = KChunk<T, D, KEYS>::NSTEP;
    f32x16 c0[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        if (c_init != nullptr) {
            c0[b] = c_init[LDS_A ? b : 0];
        } else if (init == nullptr) {
            c0[b] = f32x16{};
        } else {
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const float4 v = *reinterpret_cast<const float4*>(init + (LDS_A ? 32 * b : 0) + c_row(4 * a, lane));
                c0[b][4 * a] = v.x;
                c0[b][4 * a + 1] = v.y;
                c0[b][4 * a + 2] = v.z;
                c0[b][4 * a + 3] = v.w;
            }
        }
    }
#pragma unroll
    for (int st = 0; st < NS; ++st) {
        const typename M::frag f[2] = {rd.get(slot, 0, st), rd.get(slot, 1, st)};
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const f32x16 c = st == 0 ? c0[b] : acc[b];
            acc[b] = LDS_A ? M::mma(f[b], reg[st], c) : M::mma(reg[st], f[b], c);
        }
    }
    if constexpr (ChunkReader<T, D, KEYS>::kTable) {
        // keep the fragment reads two k-steps ahead of the products
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // LDS reads of steps 0, 1
#pragma unroll
        for (int st = 0; st < NS; ++st) {
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // products of step st
            if (st + 2 < NS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // reads of step st + 2
        }
    }
}

// chunk_mma for RS sets of 32 register rows at once: acc[s][b] is register set
// s against chunk block b, in the layout chunk_mma gives for one set.  Each
// fragment read from LDS feeds RS products and the 2 RS accumulators are
// independent chains.  The products start from acc itself with acc_init (the
// caller filled it), else from c_init, when given (the start value of each
// set: register rows, !LDS_A), else from zero.
template <typename T, int D, int KEYS, bool LDS_A, int RS>
__device__ __forceinline__ void chunk_mma_sets(f32x16 (&acc)[RS][2], const ChunkReader<T, D, KEYS>& rd,
                                               const char* slot,
                                               const typename Mma<T>::frag (&reg)[RS][KChunk<T, D, KEYS>::NSTEP],
                                               const f32x16* c_init, bool acc_init = false) {
    using M = Mma<T>;
    constexpr int NS = KChunk<T, D, KEYS>::NSTEP;
#pragma unroll
    for (int st = 0; st < NS; ++st) {
        const typename M::frag f[2] = {rd.get(slot, 0, st), rd.get(slot, 1, st)};
#pragma unroll
        for (int rs = 0; rs < RS; ++rs)
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const f32x16 c = (st > 0 || acc_init) ? acc[rs][b] : (c_init != nullptr ? c_init[rs] : f32x16{});
                acc[rs][b] = LDS_A ? M::mma(f[b], reg[rs][st], c) : M::mma(reg[rs][st], f[b], c);
            }
    }
    if constexpr (ChunkReader<T, D, KEYS>::kTable) {
        // keep the fragment reads two k-steps ahead of the products
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // LDS reads of steps 0, 1
#pragma unroll
        for (int st = 0; st < NS; ++st) {
            __builtin_amdgcn_sched_group_barrier(0x008, 2 * RS, 0);  // products of step st
            if (st + 2 < NS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // reads of step st + 2
        }
    }
}

// Running softmax denominator of one row over chunks of 32 logits per lane
// (x in acc units; sl2 turns them into log2 units).  The reference m is raised
// only when a chunk's partial sum leaves [0, 2^64] (a logit more than 64 above
// m, no reference yet, or masked logits before the first one); m is then the
// largest logit seen so far, so nothing overflows or loses precision.
struct RowSum {
    float m = -INFINITY, l = 0.0f;

    // partial sum of exp2(sl2 x - m) over the 32 values (tree order)
    __device__ __forceinline__ float part(const f32x16 (&x)[2], float sl2) const {
        f32x16 ex[2];  // the logits stay in x for a possible new reference
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i) ex[b][i] = fast_exp2(fmaf(x[b][i], sl2, -m));
        float p[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            p[e] = (ex[0][e] + ex[0][e + 4]) + (ex[0][e + 8] + ex[0][e + 12]) +
                   ((ex[1][e] + ex[1][e + 4]) + (ex[1][e + 8] + ex[1][e + 12]));
        return (p[0] + p[1]) + (p[2] + p[3]);
    }
    // the chunk's sum left [0, 2^64] (or there is no reference yet): raise
    // the reference to the largest logit seen so far and add the chunk again
    __device__ __forceinline__ void reset(const f32x16 (&x)[2], float sl2) {
        float mx = -INFINITY;
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, x[b][i]);
        const float mn = fmaxf(m, mx * sl2);
        if (mn == -INFINITY) return;
        float a = l * fast_exp2(m - mn);
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i) a += fast_exp2(fmaf(x[b][i], sl2, -mn));
        l = a;
        m = mn;
    }
    __device__ __forceinline__ void add(const f32x16 (&x)[2], float sl2) {
        const float ln = l + part(x, sl2);
        if (ln <= 0x1p64f) {  // false for inf and NaN
            l = ln;
            return;
        }
        reset(x, sl2);
    }
    // log2 of the sum, -inf when empty
    __device__ __forceinline__ float lse2() const { return (m != -INFINITY && l > 0.0f) ? m + log2f(l) : -INFINITY; }
};

// Issue order of a block with NTRANS exponentials and about twice as many other
// vector instructions: one exponential, then two other vector instructions.
// v_exp_f32 occupies the transcendental unit for 16 cycles and a wave issues in
// order, so back-to-back exponentials stall the wave while independent vector
// work waits behind them.
template <int NTRANS>
__device__ __forceinline__ void interleave_trans() {
#pragma unroll
    for (int i = 0; i < NTRANS; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x400, 1, 0);  // one transcendental
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // two other vector instructions
    }
}

// RowSum::add for RS sets at once: the exponentials and sums of every set in
// one block (one wave's vector work per chunk), then one test of all sums.
template <int RS>
__device__ __forceinline__ void row_sums_add(RowSum (&r)[RS], const f32x16 (&x)[RS][2], float sl2) {
    float ln[RS];
    bool ok = true;
#pragma unroll
    for (int rs = 0; rs < RS; ++rs) {
        ln[rs] = r[rs].l + r[rs].part(x[rs], sl2);
        ok = ok && ln[rs] <= 0x1p64f;  // false for inf and NaN
    }
    interleave_trans<32 * RS>();
    if (__builtin_expect(ok, 1)) {
#pragma unroll
        for (int rs = 0; rs < RS; ++rs) r[rs].l = ln[rs];
        return;
    }
#pragma unroll
    for (int rs = 0; rs < RS; ++rs) {
        if (ln[rs] <= 0x1p64f)
            r[rs].l = ln[rs];
        else
            r[rs].reset(x[rs], sl2);
    }
}

// Row sums of RS sets with the exponentials taken in place of the logits (x
// is destroyed), which keeps a second copy of the chunk's values out of the
// registers.  A set with no reference yet (a range's first chunk) takes the
// chunk's largest logit as its reference first, as a reset would; a set whose
// logits are all masked keeps no reference and adds 0.  Returns false, for
// the whole wave, when a sum of any lane left [0, 2^64]: ln[] then holds every
// set's new sum, lanes whose sums all stayed in range have already kept them,
// and the caller takes the chunk's logits again on every lane (a matrix-core
// product reads the fragments of every lane, so a lane left out would feed it
// stale registers) and finishes with row_sums_fix.
template <int RS>
__device__ __forceinline__ bool row_sums_try(RowSum (&r)[RS], f32x16 (&x)[RS][2], float sl2, float (&ln)[RS]) {
    bool fresh = false;
#pragma unroll
    for (int rs = 0; rs < RS; ++rs) fresh = fresh || r[rs].m == -INFINITY;
    if (__builtin_amdgcn_ballot_w64(fresh) != 0) {  // wave-uniform, rare
#pragma unroll
        for (int rs = 0; rs < RS; ++rs) {
            float mx = -INFINITY;
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, x[rs][b][i]);
            if (r[rs].m == -INFINITY) r[rs].m = mx * sl2;
        }
    }
    bool ok = true;
#pragma unroll
    for (int rs = 0; rs < RS; ++rs) {
        const float nm = r[rs].m == -INFINITY ? 0.0f : -r[rs].m;  // masked logits give 0 either way
        float p[4];
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i) x[rs][b][i] = fast_exp2(fmaf(x[rs][b][i], sl2, nm));
#pragma unroll
        for (int e = 0; e < 4; ++e)
            p[e] = (x[rs][0][e] + x[rs][0][e + 4]) + (x[rs][0][e + 8] + x[rs][0][e + 12]) +
                   ((x[rs][1][e] + x[rs][1][e + 4]) + (x[rs][1][e + 8] + x[rs][1][e + 12]));
        ln[rs] = r[rs].l + ((p[0] + p[1]) + (p[2] + p[3]));
        ok = ok && ln[rs] <= 0x1p64f;  // false for inf and NaN
    }
    interleave_trans<32 * RS>();
    if (__builtin_expect(ok, 1)) {
#pragma unroll
        for (int rs = 0; rs < RS; ++rs) r[rs].l = ln[rs];
    }
    return __builtin_amdgcn_ballot_w64(!ok) == 0;
}
// The rest of row_sums_try after a false return, with x the chunk's logits
// (on every lane): sets whose sum stayed in range keep it (again, on lanes
// that kept it already), the others raise their reference.
template <int RS>
__device__ __forceinline__ void row_sums_fix(RowSum (&r)[RS], const f32x16 (&x)[RS][2], float sl2,
                                             const float (&ln)[RS]) {
#pragma unroll
    for (int rs = 0; rs < RS; ++rs) {
        if (ln[rs] <= 0x1p64f)
            r[rs].l = ln[rs];
        else
            r[rs].reset(x[rs], sl2);
    }
}

// Sum of exp2(sl2 * x) over the 32 values a lane holds in x (in place: the
// logits are not needed again), as a tree.
__device__ __forceinline__ float exp2_sum(f32x16 (&x)[2], float sl2) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[b][i] = fast_exp2(x[b][i] * sl2);
    float part[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
        part[e] = (x[0][e] + x[0][e + 4]) + (x[0][e + 8] + x[0][e + 12]) +
                  ((x[1][e] + x[1][e + 4]) + (x[1][e + 8] + x[1][e + 12]));
    return (part[0] + part[1]) + (part[2] + part[3]);
}

}  // namespace kve
