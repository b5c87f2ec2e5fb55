// Decode attention over a compacted cache: one new query per head attends to
// the kept rows K_c[0, n), V_c[0, n) of its KV head (Algorithm 1, last step:
// decode through the keep-set; §6: a compacting implementation reads only the
// kept rows, which is where the 1 - B saving comes from).
//
// Split-K: the rows of a segment (layer, sample, KV head) are cut into splits
// of whole 128-row quanta, one workgroup each.  Every wave takes 32 rows per
// step; the query-key products run on the matrix cores (the group's query
// heads are the A rows, padded to 32, the 32 key rows the B columns) and the
// probability-weighted value sum on the vector ALU, each lane owning 16 bytes
// of a value row.  The softmax uses a lazy reference: probabilities are
// exp2(x - m) with m raised only when a logit exceeds it by more than 64 (a
// wave vote), so the common step needs no cross-lane maximum.  Each workgroup
// writes (m, l, o) per head; a second kernel merges the splits.
#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kBlk = 32;  // key rows per wave step

// Query-key fragments of one row for the 32x32 products.  The contraction
// index may be assigned to registers in any order as long as the query and the
// key rows agree; each lane reads whole 16-byte pieces.
template <typename T, int D>
struct QKFrag;

template <int D>
struct QKFrag<__bf16, D> {
    static constexpr int NSTEP = D / 16;
    typedef bf16x8 frag;
    // k-step st, lane half h: elements 16 st + 8 h .. + 8
    __device__ __forceinline__ static void load(const __bf16* row, int h, frag (&f)[NSTEP]) {
#pragma unroll
        for (int st = 0; st < NSTEP; ++st) f[st] = *reinterpret_cast<const bf16x8*>(row + 16 * st + 8 * h);
    }
    __device__ __forceinline__ static void zero(frag (&f)[NSTEP]) {
#pragma unroll
        for (int st = 0; st < NSTEP; ++st) f[st] = Mma<__bf16>::zero();
    }
};

template <int D>
struct QKFrag<float, D> {
    static constexpr int NSTEP = D / 2;
    typedef float frag;
    // k-step 4 a + b, lane half h: element 8 a + 4 h + b
    __device__ __forceinline__ static void load(const float* row, int h, frag (&f)[NSTEP]) {
#pragma unroll
        for (int a = 0; a < D / 8; ++a) {
            const float4 x = *reinterpret_cast<const float4*>(row + 8 * a + 4 * h);
            f[4 * a] = x.x;
            f[4 * a + 1] = x.y;
            f[4 * a + 2] = x.z;
            f[4 * a + 3] = x.w;
        }
    }
    __device__ __forceinline__ static void zero(frag (&f)[NSTEP]) {
#pragma unroll
        for (int st = 0; st < NSTEP; ++st) f[st] = 0.0f;
    }
};

__device__ __forceinline__ float xor_max32(float v) {
#pragma unroll
    for (int s = 1; s < 32; s <<= 1) v = fmaxf(v, __shfl_xor(v, s));
    return v;
}

__device__ __forceinline__ float xor_sum32(float v) {
#pragma unroll
    for (int s = 1; s < 32; s <<= 1) v += __shfl_xor(v, s);
    return v;
}

__device__ __forceinline__ float read_lane(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// One workgroup per (segment, split).  NH: query heads per KV head padded to
// 4 or 8.  Head h of the wave's 32x32 product sits in register h % 4 of the
// lanes of half h / 4 (rows c_row(i, lane) = 4 (lane / 32) + i for i < 4), the
// key in lane % 32.
template <typename T, int D, int NH>
__global__ __launch_bounds__(kThreads) void decode_split(const T* __restrict__ q, const T* __restrict__ kc,
                                                         const T* __restrict__ vc,
                                                         const int32_t* __restrict__ count, int G, int k_cap,
                                                         int nsplit, int split_keys, float sl2,
                                                         float* __restrict__ ws_o, float2* __restrict__ ws_ml) {
    using F = QKFrag<T, D>;
    using M = Mma<T>;
    using VP = VPiece<T>;
    constexpr int NS = F::NSTEP;
    constexpr int CW = VP::CW;        // value columns per lane
    constexpr int CPL = D / CW;       // lanes per value row
    constexpr int KPI = kWave / CPL;  // value rows per load
    constexpr int NV = kBlk / KPI;    // value loads per lane and step
    static_assert(NH == 4 || NH == 8, "4 or 8 padded heads");

    __shared__ float s_p[kWaves][kBlk][NH];
    __shared__ float s_ml[kWaves][2][NH];
    __shared__ float s_o[kWaves][NH][D];

    const int seg = blockIdx.x / nsplit;
    const int sp = blockIdx.x - seg * nsplit;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int half = lane >> 5;
    const int n = min(max(count[seg], 0), k_cap);
    const int k0 = sp * split_keys;
    const int k1 = min(n, k0 + split_keys);
    const T* ks = kc + (size_t)seg * k_cap * D;
    const T* vs = vc + (size_t)seg * k_cap * D;

    typename F::frag qf[NS];
    {
        const int h = lane & 31;
        if (h < G)
            F::load(q + ((size_t)seg * G + h) * D, half, qf);
        else
            F::zero(qf);
    }
    float m[4], l[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.0f;
    }
    float o[NH][CW];
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
        for (int c = 0; c < CW; ++c) o[h][c] = 0.0f;
    const int kq = lane / CPL, cg = lane - (lane / CPL) * CPL;

    for (int blk = k0 + wv * kBlk; blk < k1; blk += kWaves * kBlk) {
        // key fragments, then value pieces; row indices clamped into [0, n)
        typename F::frag kf[NS];
        F::load(ks + (size_t)min(blk + (lane & 31), n - 1) * D, half, kf);
        u32x4 vr[NV];
#pragma unroll
        for (int i = 0; i < NV; ++i) vr[i] = ld16(vs + (size_t)min(blk + KPI * i + kq, n - 1) * D + cg * CW);

        f32x16 acc = {};
#pragma unroll
        for (int st = 0; st < NS; ++st) acc = M::mma(qf[st], kf[st], acc);

        const bool kvalid = blk + (lane & 31) < k1;
        float x[4];
        bool raise = false;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = kvalid ? acc[i] * sl2 : -INFINITY;
            raise |= x[i] > m[i] + 64.0f;
        }
        if (__builtin_amdgcn_ballot_w64(raise) != 0) {
            // new reference: the largest of the old one and this step's logits
            float alpha[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float mn = fmaxf(m[i], xor_max32(x[i]));
                alpha[i] = mn == -INFINITY ? 1.0f : fast_exp2(m[i] - mn);
                l[i] *= alpha[i];
                m[i] = mn;
            }
#pragma unroll
            for (int h = 0; h < NH; ++h) {
                const float a = read_lane(alpha[h & 3], (h >> 2) * 32);
#pragma unroll
                for (int c = 0; c < CW; ++c) o[h][c] *= a;
            }
        }
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            p[i] = kvalid ? fast_exp2(x[i] - m[i]) : 0.0f;
            l[i] += p[i];
        }
        // every lane needs the probabilities of its value rows for every head
        if (NH == 8 || half == 0)
            *reinterpret_cast<float4*>(&s_p[wv][lane & 31][4 * half]) = make_float4(p[0], p[1], p[2], p[3]);
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int t = KPI * i + kq;
            float pp[NH];
#pragma unroll
            for (int a = 0; a < NH / 4; ++a) {
                const float4 v4 = *reinterpret_cast<const float4*>(&s_p[wv][t][4 * a]);
                pp[4 * a] = v4.x;
                pp[4 * a + 1] = v4.y;
                pp[4 * a + 2] = v4.z;
                pp[4 * a + 3] = v4.w;
            }
            float vf[CW];
            VP::to_f(vr[i], vf);
#pragma unroll
            for (int h = 0; h < NH; ++h)
#pragma unroll
                for (int c = 0; c < CW; ++c) o[h][c] = fmaf(pp[h], vf[c], o[h][c]);
        }
        __builtin_amdgcn_wave_barrier();
    }

    // the wave's sums: l over the 32 key lanes of each half, o over the lanes
    // that share value columns
#pragma unroll
    for (int i = 0; i < 4; ++i) l[i] = xor_sum32(l[i]);
#pragma unroll
    for (int s = CPL; s < kWave; s <<= 1)
#pragma unroll
        for (int h = 0; h < NH; ++h)
#pragma unroll
            for (int c = 0; c < CW; ++c) o[h][c] += __shfl_xor(o[h][c], s);
    if ((lane & 31) == 0 && (NH == 8 || half == 0)) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            s_ml[wv][0][4 * half + i] = m[i];
            s_ml[wv][1][4 * half + i] = l[i];
        }
    }
    if (kq == 0) {
#pragma unroll
        for (int h = 0; h < NH; ++h)
#pragma unroll
            for (int c = 0; c < CW; ++c) s_o[wv][h][cg * CW + c] = o[h][c];
    }
    __syncthreads();
    // merge the waves' partial results of this split
    for (int e = threadIdx.x; e < G * D; e += kThreads) {
        const int h = e / D, c = e - (e / D) * D;
        float mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, s_ml[w][0][h]);
        float lt = 0.0f, ot = 0.0f;
        if (mx != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                const float a = fast_exp2(s_ml[w][0][h] - mx);
                lt = fmaf(a, s_ml[w][1][h], lt);
                ot = fmaf(a, s_o[w][h][c], ot);
            }
        }
        ws_o[((size_t)blockIdx.x * G + h) * D + c] = ot;
        if (c == 0) ws_ml[(size_t)blockIdx.x * G + h] = make_float2(mx, lt);
    }
}

// One wave per (segment, head): merge the splits and normalise.
template <int D>
__global__ __launch_bounds__(kThreads) void decode_combine(const float* __restrict__ ws_o,
                                                           const float2* __restrict__ ws_ml, int G, int nsplit,
                                                           int n_rows, float* __restrict__ out) {
    const int r = blockIdx.x * kWaves + (int)(threadIdx.x / kWave);
    if (r >= n_rows) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int seg = r / G, h = r - (r / G) * G;
    constexpr int CPT = D / kWave;
    const size_t base = (size_t)seg * nsplit;
    float mx = -INFINITY;
    for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, ws_ml[(base + s) * G + h].x);
    float lt = 0.0f, ot[CPT];
#pragma unroll
    for (int c = 0; c < CPT; ++c) ot[c] = 0.0f;
    if (mx != -INFINITY) {
        for (int s = 0; s < nsplit; ++s) {
            const float2 ml = ws_ml[(base + s) * G + h];
            const float a = fast_exp2(ml.x - mx);
            lt = fmaf(a, ml.y, lt);
            const float* os = ws_o + ((base + s) * G + h) * D + lane * CPT;
#pragma unroll
            for (int c = 0; c < CPT; ++c) ot[c] = fmaf(a, os[c], ot[c]);
        }
    }
#pragma unroll
    for (int c = 0; c < CPT; ++c) out[(size_t)r * D + lane * CPT + c] = lt > 0.0f ? ot[c] / lt : 0.0f;
}

template <typename T, int D, int NH>
hipError_t run_decode(const void* q, const void* kc, const void* vc, const int32_t* count, int L, int B,
                      int Hq, int Hkv, int k_cap, float scale, float* out, void* ws, hipStream_t st) {
    const DecodePlan p = decode_plan(L, B, Hq, Hkv, k_cap, D);
    char* w = static_cast<char*>(ws);
    float* wo = reinterpret_cast<float*>(w + p.off_o);
    float2* wml = reinterpret_cast<float2*>(w + p.off_ml);
    hipLaunchKernelGGL((decode_split<T, D, NH>), dim3((unsigned)((size_t)p.segs * p.nsplit)), dim3(kThreads), 0,
                       st, static_cast<const T*>(q), static_cast<const T*>(kc), static_cast<const T*>(vc), count,
                       p.G, k_cap, p.nsplit, p.split_keys, scale * kLog2e, wo, wml);
    const int rows = p.segs * p.G;
    hipLaunchKernelGGL((decode_combine<D>), dim3((unsigned)((rows + kWaves - 1) / kWaves)), dim3(kThreads), 0, st,
                       wo, wml, p.G, p.nsplit, rows, out);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t run_decode_g(const void* q, const void* kc, const void* vc, const int32_t* count, int L, int B,
                        int Hq, int Hkv, int k_cap, float scale, float* out, void* ws, hipStream_t st) {
    if (Hq / Hkv <= 4) return run_decode<T, D, 4>(q, kc, vc, count, L, B, Hq, Hkv, k_cap, scale, out, ws, st);
    return run_decode<T, D, 8>(q, kc, vc, count, L, B, Hq, Hkv, k_cap, scale, out, ws, st);
}

}  // namespace

hipError_t launch_decode(const void* q, const void* kc, const void* vc, const int32_t* count, int dtype, int L,
                         int B, int Hq, int Hkv, int k_cap, int d, float scale, float* out, void* ws,
                         hipStream_t st) {
    if (dtype == 0) {
        if (d == 128) return run_decode_g<__bf16, 128>(q, kc, vc, count, L, B, Hq, Hkv, k_cap, scale, out, ws, st);
        return run_decode_g<__bf16, 64>(q, kc, vc, count, L, B, Hq, Hkv, k_cap, scale, out, ws, st);
    }
    if (d == 128) return run_decode_g<float, 128>(q, kc, vc, count, L, B, Hq, Hkv, k_cap, scale, out, ws, st);
    return run_decode_g<float, 64>(q, kc, vc, count, L, B, Hq, Hkv, k_cap, scale, out, ws, st);
}

}  // namespace kve
