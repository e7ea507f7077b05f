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

// Sum of each of 16 per-lane values over the 64 lanes of a wave, by halving
// exchanges: afterwards lane l holds the total of value index
// 8 b5 + 4 b4 + 2 b3 + b2 (b_k = bit k of l).  17 exchanges instead of 96.
__device__ __forceinline__ float wave_sum16(const float (&p)[16], int lane) {
    const bool h5 = (lane >> 5) & 1, h4 = (lane >> 4) & 1, h3 = (lane >> 3) & 1, h2 = (lane >> 2) & 1;
    float a8[8], a4[4], a2[2];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const float send = h5 ? p[k] : p[8 + k];
        a8[k] = (h5 ? p[8 + k] : p[k]) + __shfl_xor(send, 32, 64);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float send = h4 ? a8[k] : a8[4 + k];
        a4[k] = (h4 ? a8[4 + k] : a8[k]) + __shfl_xor(send, 16, 64);
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const float send = h3 ? a4[k] : a4[2 + k];
        a2[k] = (h3 ? a4[2 + k] : a4[k]) + __shfl_xor(send, 8, 64);
    }
    float a1 = (h2 ? a2[1] : a2[0]) + __shfl_xor(h2 ? a2[0] : a2[1], 4, 64);
    a1 += __shfl_xor(a1, 2, 64);
    a1 += __shfl_xor(a1, 1, 64);
    return a1;
}

// u: this thread's values of the row, chunk i covers columns 4 (tid + 256 i) .. +3
// (chunks past the row's end may hold anything).  Must be called by all 256
// threads of the block (it synchronizes).  The loads of a chunk's 16 A rows
// are unconditional (ranks past rs re-read row rs - 1 and are dropped) so that
// they are in flight together.
//
// With several blocks per row (slice of nslice), block `slice` takes every
// nslice-th group of 16 ranks (targets in order) and only slice 0 writes the
// zero columns.
template <typename T, int MAXC>
__device__ __forceinline__ void row_shrink(const RowShrink& sh, int m, int d, const f32x4 (&u)[MAXC],
                                           float (*red)[16], int slice = 0, int nslice = 1) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nc = d / 4;
    const int slot = sh.row_slot[m];
    T* zr = (T*)sh.Z + (int64_t)m * 4 * sh.kw;
    // zero every column outside the row's own slot block of an active target
    if (slice == 0)
        for (int c = tid; c < 3 * sh.kw; c += 256) {
            const int t = c / sh.kw, cc = c % sh.kw;
            const bool own = slot >= 0 && ((sh.mask >> t) & 1u) && cc >= slot * sh.rs && cc < (slot + 1) * sh.rs;
            if (!own) zr[c] = (T)0.f;
        }
    if (slot < 0) return;  // uniform across the block
    const float scale = sh.slot_scale[slot];
    const T* A = (const T*)sh.Acat;
    const int o_lane = 8 * ((lane >> 5) & 1) + 4 * ((lane >> 4) & 1) + 2 * ((lane >> 3) & 1) + ((lane >> 2) & 1);
    int group = 0;
    for (int t = 0; t < 3; ++t) {
        if (!((sh.mask >> t) & 1u)) continue;
        for (int j0 = 0; j0 < sh.rs; j0 += 16) {
            if (group++ % nslice != slice) continue;  // uniform across the block
            const T* rows[16];
#pragma unroll
            for (int o = 0; o < 16; ++o)
                rows[o] = A + (int64_t)(t * sh.kw + slot * sh.rs + min(j0 + o, sh.rs - 1)) * d;
            float part[16];
#pragma unroll
            for (int o = 0; o < 16; ++o) part[o] = 0.f;
#pragma unroll
            for (int i = 0; i < MAXC; ++i) {
                if (256 * i >= nc) break;  // uniform
                const int c = tid + 256 * i;
                const bool valid = c < nc;
                const int cc = valid ? c : 0;
                u32x2 raw[16];
#pragma unroll
                for (int o = 0; o < 16; ++o) raw[o] = *(const u32x2*)(rows[o] + 4 * cc);
                float uu[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) uu[r] = valid ? u[i][r] : 0.f;
#pragma unroll
                for (int o = 0; o < 16; ++o) {
                    T a4[4];
                    __builtin_memcpy(a4, &raw[o], 8);
                    part[o] += uu[0] * (float)a4[0] + uu[1] * (float)a4[1] + uu[2] * (float)a4[2] +
                               uu[3] * (float)a4[3];
                }
            }
            const float tot = wave_sum16(part, lane);
            lds_barrier();  // previous use of red finished
            if ((lane & 3) == 0) red[wave][o_lane] = tot;
            lds_barrier();
            if (tid < 16 && j0 + tid < sh.rs) {
                const float zsum = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
                zr[t * sh.kw + slot * sh.rs + j0 + tid] = (T)(scale * zsum);
            }
        }
    }
}

}  // namespace pb
