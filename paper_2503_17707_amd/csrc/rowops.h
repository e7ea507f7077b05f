// Row-wise LoRA shrink fused into the kernels that produce a LayerNorm row.
//
// For token m with adapter slot s >= 0, and each target t in {q, k, v} of the
// mask, Z[m, t*kw + s*rs + j] = dt(scale_s * sum_k u[m, k] * Acat[t][s*rs + j][k])
// for j < rs (ranks past the adapter's own are zero rows of Acat), and every
// other column of Z[m, 0 .. 3 kw) is 0, exactly the layout the shrink GEMM
// writes.  u enters rounded to dt, as it enters the projection GEMM.
#pragma once

#include "common.h"

namespace pb {

struct RowShrink {
    const void* Acat;        // this layer's [4][kw][d] A slots (dt); NULL = no shrink
    const int32_t* row_slot; // [M]
    const float* slot_scale; // [16]
    void* Z;                 // [M][4 kw] (dt)
    int rs, kw;
    uint32_t mask;           // targets q=1, k=2, v=4
};

// One LayerNorm output before rounding: (v - mean) rstd g + b, with the
// rounding steps spelled out (product, then one fused multiply-add) so that
// every kernel that normalizes a row gets the same bits, whatever the
// compiler would contract.  The empty asm keeps the result an fp32 value:
// otherwise a later conversion to fp16 may be folded into a mixed-precision
// multiply-add that rounds once to fp16 instead of to fp32 and then to fp16.
__device__ __forceinline__ float ln_apply(float v, float mean, float rstd, float g, float b) {
    float y = __builtin_fmaf((v - mean) * rstd, g, b);
    asm("" : "+v"(y));
    return y;
}

// 1 / sqrt(var + eps) from the block sum of squared deviations, the variance
// rounded inside one fused multiply-add (q inv_d + eps)
__device__ __forceinline__ float ln_rstd(float qsum, float inv_d, float eps) {
    return 1.0f / sqrtf(__builtin_fmaf(qsum, inv_d, eps));
}

// Sum over the 256 threads of a block (4 waves); red holds 4 floats.
__device__ __forceinline__ float block_sum256(float v, float* red) {
    v = wave_sum(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    lds_barrier();  // previous use of red finished
    if (lane == 0) red[wave] = v;
    lds_barrier();
    return (red[0] + red[1]) + (red[2] + red[3]);
}

// LayerNorm of one row of d = 4 nc values held by the 256 threads of a block
// as float4 chunks (chunk i of a thread = columns 4 (tid + 256 i) .. +3; sum =
// this thread's sum of its values): out = LN(v) * g + b with fp32 statistics
// (biased variance), written as dt, or fp32 when OUT_F32.  For dt
// output v is left holding the values rounded to dt, as the next GEMM reads them.
// out_row NULL: nothing is written (v is still updated).
template <typename T, int MAXC, bool OUT_F32>
__device__ __forceinline__ void row_layernorm(f32x4 (&v)[MAXC], float sum, int nc, const T* g, const T* b,
                                              void* out_row, float eps, float* red) {
#pragma clang fp contract(off)  // only the fused multiply-adds written out below
    const int tid = threadIdx.x;
    // narrow rows: g and b preloaded (their latency hides behind the
    // reductions); wide rows: loaded at the end, their registers would cost
    // rows in flight
    constexpr bool PRE = MAXC <= 4;
    u32x2 graw[PRE ? MAXC : 1], braw[PRE ? MAXC : 1];
    if (PRE) {
#pragma unroll
        for (int i = 0; i < MAXC; ++i) {
            const int c = tid + 256 * i;
            if (c < nc) {
                graw[PRE ? i : 0] = *(const u32x2*)(g + 4 * c);
                braw[PRE ? i : 0] = *(const u32x2*)(b + 4 * c);
            }
        }
    }
    const float inv_d = 1.0f / (float)(4 * nc);
    const float mean = block_sum256(sum, red) * inv_d;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i)
        if (tid + 256 * i < nc)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float t = v[i][r] - mean;
                q = __builtin_fmaf(t, t, q);
            }
    const float rstd = ln_rstd(block_sum256(q, red), inv_d, eps);
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
        const int c = tid + 256 * i;
        if (c < nc) {
            T ga[4], ba[4];
            const u32x2 gr = PRE ? graw[PRE ? i : 0] : *(const u32x2*)(g + 4 * c);
            const u32x2 br = PRE ? braw[PRE ? i : 0] : *(const u32x2*)(b + 4 * c);
            __builtin_memcpy(ga, &gr, 8);
            __builtin_memcpy(ba, &br, 8);
            float y[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) y[r] = ln_apply(v[i][r], mean, rstd, (float)ga[r], (float)ba[r]);
            if (OUT_F32) {
                if (out_row) *(f32x4*)((float*)out_row + 4 * c) = f32x4{y[0], y[1], y[2], y[3]};
            } else {
                if (out_row) *(u32x2*)((T*)out_row + 4 * c) = pack4<T>(y[0], y[1], y[2], y[3]);
#pragma unroll
                for (int r = 0; r < 4; ++r) v[i][r] = (float)(T)y[r];
            }
        }
    }
}

// Sum over the 64 lanes of each of M (a power of two up to 32) per-lane
// values by halving exchanges: afterwards lane l holds the total of value
// index l >> (6 - log2 M) (for M = 16: 8 b5 + 4 b4 + 2 b3 + b2, b_k = bit k
// of l); M - 1 + 6 - log2 M exchanges instead of 6 M.  Each step keeps the
// half it still needs in a fresh array, so the values already exchanged are
// dead (fewer live registers than halving in place).
template <int M, int D>
__device__ __forceinline__ float wave_sum_halves(const float (&p)[M], int lane) {
    if constexpr (M == 1) {
        float a = p[0];
#pragma unroll
        for (int e = D; e > 0; e >>= 1) a += __shfl_xor(a, e, 64);
        return a;
    } else {
        constexpr int n = M / 2;
        const bool up = (lane & D) != 0;
        float q[n];
#pragma unroll
        for (int k = 0; k < n; ++k) {
            const float send = up ? p[k] : p[n + k];
            q[k] = (up ? p[n + k] : p[k]) + __shfl_xor(send, D, 64);
        }
        return wave_sum_halves<n, D / 2>(q, lane);
    }
}

template <int M>
__device__ __forceinline__ float wave_sum_multi(const float (&p)[M], int lane) {
    static_assert(M >= 1 && M <= 32 && (M & (M - 1)) == 0, "power of two up to 32");
    return wave_sum_halves<M, 32>(p, lane);
}

// u: this thread's values of the row, chunk i covers columns 4 (tid + 256 i) .. +3
// (chunks past the row's end may hold anything).  Must be called by all 256
// threads of the block (it synchronizes).  Ranks go in groups of G (4, 8 or
// 16); the loads of a chunk's G A rows are unconditional (ranks past rs
// re-read row rs - 1 and are dropped) so that they are in flight together.
//
// With several blocks per row (slice of nslice), block `slice` takes every
// nslice-th group of G ranks (targets in order) and only slice 0 writes the
// zero columns.
// The A words of the first rank group a block takes, with the row's slot and
// scale, loaded before the row's LayerNorm so that their latency overlaps it (for
// launches of few rows: it costs MAXC x G x 2 registers per thread).
template <int MAXC, int G>
struct ShrinkAhead {
    int slot;            // the row's adapter slot (< 0: none)
    float scale;         // its LoRA scale
    int t, j0;           // the block's first group: target and first rank (t < 0: none)
    u32x2 raw[MAXC][G];  // its A words at this thread's chunks
};

// Issue the loads of `a` (block `slice` of `nslice` on row m); `slot` is the
// row's slot, loaded by the caller ahead of its own row loads.
template <typename T, int MAXC, int G>
__device__ __forceinline__ void shrink_ahead(const RowShrink& sh, int d, int slot, int slice, int nslice,
                                             ShrinkAhead<MAXC, G>& a) {
    a.slot = slot;
    a.t = -1;
    a.j0 = 0;
    if (slot < 0) return;
    a.scale = sh.slot_scale[slot];
    int group = 0;  // groups in (target, first rank) order; the block's first is number `slice`
    for (int t = 0; t < 3 && a.t < 0; ++t) {
        if (!((sh.mask >> t) & 1u)) continue;
        for (int j0 = 0; j0 < sh.rs; j0 += G)
            if (group++ == slice) {
                a.t = t;
                a.j0 = j0;
                break;
            }
    }
    if (a.t < 0) return;  // uniform across the block
    const T* A = (const T*)sh.Acat;
    const int nc = d / 4;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
        if (256 * i >= nc) break;  // uniform
        const int c = threadIdx.x + 256 * i;
        const int cc = c < nc ? c : 0;
#pragma unroll
        for (int o = 0; o < G; ++o)
            a.raw[i][o] = *(const u32x2*)(A + (int64_t)(a.t * sh.kw + slot * sh.rs + min(a.j0 + o, sh.rs - 1)) * d +
                                          4 * cc);
    }
}

// u: this thread's values of the row, chunk i covers columns 4 (tid + 256 i) .. +3
// (chunks past the row's end may hold anything).  Must be called by all 256
// threads of the block (it synchronizes).  Ranks go in groups of G (4, 8 or
// 16); the loads of a chunk's G A rows are unconditional (ranks past rs
// re-read row rs - 1 and are dropped) so that they are in flight together.
//
// With several blocks per row (slice of nslice), block `slice` takes every
// nslice-th group of G ranks (targets in order) and only slice 0 writes the
// zero columns.  `ahead` (may be null): the slot, its scale and the first
// group's A words, already loaded by shrink_ahead.
template <typename T, int MAXC, int G = 16>
__device__ __forceinline__ void row_shrink(const RowShrink& sh, int m, int d, const f32x4 (&u)[MAXC],
                                           float (*red)[16], int slice = 0, int nslice = 1,
                                           const ShrinkAhead<MAXC, G>* ahead = nullptr) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nc = d / 4;
    const int slot = ahead ? ahead->slot : sh.row_slot[m];
    T* zr = (T*)sh.Z + (int64_t)m * 4 * sh.kw;
    // zero every column outside the row's own slot block of an active target
    if (slice == 0)
        for (int c = tid; c < 3 * sh.kw; c += 256) {
            const int t = c / sh.kw, cc = c % sh.kw;
            const bool own = slot >= 0 && ((sh.mask >> t) & 1u) && cc >= slot * sh.rs && cc < (slot + 1) * sh.rs;
            if (!own) zr[c] = (T)0.f;
        }
    if (slot < 0) return;  // uniform across the block
    const float scale = ahead ? ahead->scale : sh.slot_scale[slot];
    const T* A = (const T*)sh.Acat;
    static_assert(G == 4 || G == 8 || G == 16, "rank groups of 4, 8 or 16");
    constexpr int LG = G == 4 ? 2 : G == 8 ? 3 : 4;
    int group = 0;
    for (int t = 0; t < 3; ++t) {
        if (!((sh.mask >> t) & 1u)) continue;
        for (int j0 = 0; j0 < sh.rs; j0 += G) {
            if (group++ % nslice != slice) continue;  // uniform across the block
            const bool pre = ahead && t == ahead->t && j0 == ahead->j0;  // uniform
            const T* rows[G];
#pragma unroll
            for (int o = 0; o < G; ++o)
                rows[o] = A + (int64_t)(t * sh.kw + slot * sh.rs + min(j0 + o, sh.rs - 1)) * d;
            float part[G];
#pragma unroll
            for (int o = 0; o < G; ++o) part[o] = 0.f;
#pragma unroll
            for (int i = 0; i < MAXC; ++i) {
                if (256 * i >= nc) break;  // uniform
                const int c = tid + 256 * i;
                const bool valid = c < nc;
                const int cc = valid ? c : 0;
                u32x2 raw[G];
#pragma unroll
                for (int o = 0; o < G; ++o) raw[o] = pre ? ahead->raw[i][o] : *(const u32x2*)(rows[o] + 4 * cc);
                float uu[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) uu[r] = valid ? u[i][r] : 0.f;
#pragma unroll
                for (int o = 0; o < G; ++o) {
                    T a4[4];
                    __builtin_memcpy(a4, &raw[o], 8);
                    part[o] += uu[0] * (float)a4[0] + uu[1] * (float)a4[1] + uu[2] * (float)a4[2] +
                               uu[3] * (float)a4[3];
                }
            }
            const float tot = wave_sum_multi<G>(part, lane);
            lds_barrier();  // previous use of red finished
            if ((lane & ((64 >> LG) - 1)) == 0) red[wave][lane >> (6 - LG)] = tot;
            lds_barrier();
            if (tid < G && j0 + tid < sh.rs) {
                const float zsum = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
                zr[t * sh.kw + slot * sh.rs + j0 + tid] = (T)(scale * zsum);
            }
        }
    }
}

}  // namespace pb
