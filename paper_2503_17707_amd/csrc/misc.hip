// Memory-bound kernels of the prefill: embedding, LayerNorm, LM head, argmax
// and the LoRA slot packing.  All read and write with 16-byte vectors.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace pb {

thread_local LaunchTiming g_launch_timing = {nullptr, nullptr};

namespace {

// ---- embedding: OPT learned absolute positions, no offset -------------------
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const int32_t* __restrict__ tok,
                                                   const T* __restrict__ E,
                                                   const T* __restrict__ P,
                                                   float* __restrict__ x, int T_len, int d,
                                                   const int32_t* __restrict__ pos0) {
    const int row = blockIdx.x;
    const int t = *pos0 + row % T_len;
    const T* e = E + (int64_t)tok[row] * d;
    const T* pp = P + (int64_t)t * d;
    float* xr = x + (int64_t)row * d;
    for (int c = threadIdx.x * 8; c < d; c += 256 * 8) {
        const u32x4 ev = *(const u32x4*)(e + c);
        const u32x4 pv = *(const u32x4*)(pp + c);
        T ea[8], pa[8];
        __builtin_memcpy(ea, &ev, 16);
        __builtin_memcpy(pa, &pv, 16);
        f32x4 lo, hi;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            lo[i] = (float)ea[i] + (float)pa[i];
            hi[i] = (float)ea[4 + i] + (float)pa[4 + i];
        }
        *(f32x4*)(xr + c) = lo;
        *(f32x4*)(xr + c + 4) = hi;
    }
}

// ---- LayerNorm: one 256-thread block per row, values kept in registers ------
constexpr int LN_MAXC = 16;  // float4 chunks per thread: d <= 256 * 4 * 16

// SHRINK: the row's LoRA shrink rides along (compiled only where it is used,
// since its registers would lower the occupancy of the plain kernel)
template <typename T, bool OUT_F32, int MAXC, bool SHRINK>
__global__ __launch_bounds__(256) void layernorm_kernel(const float* __restrict__ x,
                                                       int64_t in_mul, int64_t in_add,
                                                       const T* __restrict__ g,
                                                       const T* __restrict__ b, void* out,
                                                       int d, float eps, RowShrink sh) {
    __shared__ float red[4];
    const int row = blockIdx.x;
    const float* xr = x + ((int64_t)row * in_mul + in_add) * d;
    const int nc = d / 4;
    f32x4 v[MAXC];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
        const int c = threadIdx.x + 256 * i;
        if (c < nc) {
            v[i] = *(const f32x4*)(xr + 4 * c);
            s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
        }
    }
    // with gridDim.y > 1 every block of the row normalizes it, block 0 writes
    // it, and the blocks share the row's LoRA shrink
    void* orow = OUT_F32 ? (void*)((float*)out + (int64_t)row * d) : (void*)((T*)out + (int64_t)row * d);
    row_layernorm<T, MAXC, OUT_F32>(v, s, nc, g, b, blockIdx.y == 0 ? orow : nullptr, eps, red);
    if (!OUT_F32 && SHRINK) {
        __shared__ float red16[4][16];
        row_shrink<T, MAXC>(sh, row, d, v, red16, (int)blockIdx.y, (int)gridDim.y);
    }
}

// ---- LM head + argmax partials ----------------------------------------------
// logits[b, v] = z[b] . E[v] for NB sequences at once; each wave takes 8
// vocabulary rows at a time (lanes split the model width into 16-byte chunks),
// and each block also writes, per sequence, the (max, lowest index) of the
// rows it covered, so the final argmax only scans one partial per block.
#ifndef PB_LM_NT
#define PB_LM_NT 1  // embedding rows read with non-temporal loads (44.1 -> 38.6 us at OPT-1.3B)
#endif
constexpr int LM_ROWS = 8;                      // rows per wave pass
constexpr int LM_BLOCK_ROWS = 4 * 2 * LM_ROWS;  // 4 waves x 2 passes

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

template <typename T, int NB>
__global__ __launch_bounds__(256) void lm_head_kernel(const float* __restrict__ z, int b0,
                                                     const T* __restrict__ E, int V, int d,
                                                     float* __restrict__ logits,
                                                     float* __restrict__ pval,
                                                     int* __restrict__ pidx, int nblk) {
    __shared__ float sv[4][NB];
    __shared__ int si[4][NB];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    float best[NB];
    int bidx[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        best[j] = -INFINITY;
        bidx[j] = 0x7fffffff;
    }
    for (int pass = 0; pass < 2; ++pass) {
        const int v0 = blockIdx.x * LM_BLOCK_ROWS + (pass * 4 + wave) * LM_ROWS;
        if (v0 >= V) break;
        float acc[LM_ROWS][NB];
#pragma unroll
        for (int r = 0; r < LM_ROWS; ++r)
#pragma unroll
            for (int j = 0; j < NB; ++j) acc[r][j] = 0.f;
        for (int c = lane * 8; c < d; c += 64 * 8) {
            u32x4 ev[LM_ROWS];
#pragma unroll
            for (int r = 0; r < LM_ROWS; ++r) {
                const u32x4* src = (const u32x4*)(E + (int64_t)min(v0 + r, V - 1) * d + c);
#if PB_LM_NT
                ev[r] = __builtin_nontemporal_load(src);  // streamed once: no reuse to keep in cache
#else
                ev[r] = *src;
#endif
            }
            float zb[NB][8];
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const f32x4 a = *(const f32x4*)(z + (int64_t)(b0 + j) * d + c);
                const f32x4 bq = *(const f32x4*)(z + (int64_t)(b0 + j) * d + c + 4);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    zb[j][e] = a[e];
                    zb[j][4 + e] = bq[e];
                }
            }
#pragma unroll
            for (int r = 0; r < LM_ROWS; ++r) {
                T ea[8];
                __builtin_memcpy(ea, &ev[r], 16);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float w = (float)ea[e];
#pragma unroll
                    for (int j = 0; j < NB; ++j) acc[r][j] += w * zb[j][e];
                }
            }
        }
#pragma unroll
        for (int r = 0; r < LM_ROWS; ++r)
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const float t = wave_sum(acc[r][j]);
                const int v = v0 + r;
                if (v < V) {
                    if (lane == 0) logits[(int64_t)(b0 + j) * V + v] = t;
                    if (better(t, v, best[j], bidx[j])) {
                        best[j] = t;
                        bidx[j] = v;
                    }
                }
            }
    }
    if (lane == 0)
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            sv[wave][j] = best[j];
            si[wave][j] = bidx[j];
        }
    __syncthreads();
    if (threadIdx.x < NB) {
        const int j = threadIdx.x;
        float bb = sv[0][j];
        int ii = si[0][j];
        for (int w = 1; w < 4; ++w)
            if (better(sv[w][j], si[w][j], bb, ii)) {
                bb = sv[w][j];
                ii = si[w][j];
            }
        pval[(int64_t)(b0 + j) * nblk + blockIdx.x] = bb;
        pidx[(int64_t)(b0 + j) * nblk + blockIdx.x] = ii;
    }
}

// ---- argmax over the per-block partials: one block per sequence ------------
__global__ __launch_bounds__(256) void argmax_final_kernel(const float* __restrict__ pval,
                                                          const int* __restrict__ pidx, int nblk,
                                                          int32_t* __restrict__ tok) {
    __shared__ float sv[4];
    __shared__ int si[4];
    const int b = blockIdx.x;
    float best = -INFINITY;
    int bi = 0x7fffffff;
    for (int i = threadIdx.x; i < nblk; i += 256) {
        const float x = pval[(int64_t)b * nblk + i];
        const int xi = pidx[(int64_t)b * nblk + i];
        if (better(x, xi, best, bi)) {
            best = x;
            bi = xi;
        }
    }
    for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(best, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (better(ov, oi, best, bi)) {
            best = ov;
            bi = oi;
        }
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) {
        sv[wave] = best;
        si[wave] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float bb = sv[0];
        int ii = si[0];
        for (int w = 1; w < 4; ++w)
            if (better(sv[w], si[w], bb, ii)) {
                bb = sv[w];
                ii = si[w];
            }
        tok[b] = (ii == 0x7fffffff || !(bb > -INFINITY)) ? -1 : ii;
    }
}

// ---- LoRA slot packing -----------------------------------------------------
// grid (L, 4 targets, 2 parts); part 0 writes Acat[l][t][slot*rs + j][:],
// part 1 writes Bcat[l][t][n][slot*rs + j].
template <typename T>
__global__ __launch_bounds__(256) void lora_pack_kernel(const T* __restrict__ staging,
                                                       size_t staging_layer_elems, int d, int r,
                                                       uint32_t mask, int slot, int rs, int kw,
                                                       T* __restrict__ Acat,
                                                       T* __restrict__ Bcat) {
    const int l = blockIdx.x, t = blockIdx.y, part = blockIdx.z;
    const bool present = (mask >> t) & 1u;
    // position of target t in the staged blob: targets before it that are present
    int idx = 0;
    for (int u = 0; u < t; ++u) idx += (mask >> u) & 1u;
    const T* A = staging + (size_t)l * staging_layer_elems + (size_t)idx * 2 * r * d;
    const T* Bm = A + (size_t)r * d;
    const T zero = (T)0.f;
    if (part == 0) {
        T* dst = Acat + ((size_t)l * 4 + t) * (size_t)kw * d + (size_t)slot * rs * d;
        for (int i = threadIdx.x; i < rs * d; i += 256) {
            const int j = i / d;
            dst[i] = (present && j < r) ? A[i] : zero;
        }
    } else {
        T* dst = Bcat + ((size_t)l * 4 + t) * (size_t)d * kw + (size_t)slot * rs;
        for (int i = threadIdx.x; i < d * rs; i += 256) {
            const int n = i / rs, j = i % rs;
            dst[(size_t)n * kw + j] = (present && j < r) ? Bm[(size_t)n * r + j] : zero;
        }
    }
}


// ---- merged LoRA: W_t += s * B_t A_t in place ------------------------------
// Thread (row n, columns 8c .. 8c+7) of target weight W [d, d]: the rank-rs
// product of the slot's B rows (Bcat [d][kw], columns slot*rs ..) and A
// columns (Acat [kw][d], rows slot*rs ..) in fp32, ranks in order, then one
// rounding of W + s * product to dt.
template <typename T>
__global__ __launch_bounds__(256) void lora_merge_kernel(T* __restrict__ W, const T* __restrict__ Acat,
                                                        const T* __restrict__ Bcat, int d, int kw,
                                                        int rs, int slot, float scale) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int per_row = d / 8;
    if (i >= (int64_t)d * per_row) return;
    const int n = (int)(i / per_row), c = (int)(i % per_row) * 8;
    float acc[8] = {};
    const T* brow = Bcat + (int64_t)n * kw + (int64_t)slot * rs;
    for (int j = 0; j < rs; ++j) {
        const float b = (float)brow[j];
        const u32x4 araw = *(const u32x4*)(Acat + ((int64_t)slot * rs + j) * d + c);
        T a[8];
        __builtin_memcpy(a, &araw, 16);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += b * (float)a[e];
    }
    T* w = W + (int64_t)n * d + c;
    const u32x4 wraw = *(const u32x4*)w;
    T wv[8];
    __builtin_memcpy(wv, &wraw, 16);
#pragma unroll
    for (int e = 0; e < 8; ++e) wv[e] = (T)((float)wv[e] + scale * acc[e]);
    u32x4 out;
    __builtin_memcpy(&out, wv, 16);
    *(u32x4*)w = out;
}
}  // namespace

hipError_t launch_embed(int dtype, const int32_t* tok, const void* E, const void* P, float* x,
                        int n_rows, int T_len, int d, const int32_t* pos0, hipStream_t s) {
    if (n_rows <= 0) return hipSuccess;
    if (dtype == 1)
        PB_LAUNCH(embed_kernel<_Float16>, dim3(n_rows), dim3(256), 0, s, tok,
                           (const _Float16*)E, (const _Float16*)P, x, T_len, d, pos0);
    else
        PB_LAUNCH(embed_kernel<__bf16>, dim3(n_rows), dim3(256), 0, s, tok,
                           (const __bf16*)E, (const __bf16*)P, x, T_len, d, pos0);
    return hipGetLastError();
}

hipError_t launch_layernorm(int dtype, const float* x, int64_t in_mul, int64_t in_add,
                            const void* g, const void* b, void* out, bool out_f32, int rows,
                            int d, float eps, hipStream_t s, const RowShrink* shp) {
    if (rows <= 0) return hipSuccess;
    if (d % 4 || d > 256 * 4 * LN_MAXC) return hipErrorInvalidValue;
    RowShrink sh{};
    if (shp && !out_f32) sh = *shp;
    // a few rows (decode steps): the row's shrink groups of 16 ranks go to
    // blocks of their own, so that the A reads spread over several CUs
    int slices = 1;
    if (sh.Acat && rows <= 8)
        slices = std::max(1, __builtin_popcount(sh.mask & 7u) * ((sh.rs + 15) / 16));
#define PB_LN2(T, F, C, SH)                                                                        \
    PB_LAUNCH((layernorm_kernel<T, F, C, SH>), dim3(rows, slices), dim3(256), 0, s, x, in_mul,      \
              in_add, (const T*)g, (const T*)b, out, d, eps, sh)
#define PB_LN1(T, F, C)                                                                            \
    do {                                                                                           \
        if (!F && sh.Acat) PB_LN2(T, false, C, true);                                              \
        else PB_LN2(T, F, C, false);                                                               \
    } while (0)
    // chunks per thread fitted to d: registers decide how many rows a CU
    // keeps in flight, and the kernel is bound by the latency of its rows
#define PB_LN(T, F)                                                                                \
    do {                                                                                           \
        if (d <= 2048) PB_LN1(T, F, 2);                                                            \
        else if (d <= 4096) PB_LN1(T, F, 4);                                                       \
        else if (d <= 5120) PB_LN1(T, F, 5);                                                       \
        else if (d <= 8192) PB_LN1(T, F, 8);                                                       \
        else if (d <= 9216) PB_LN1(T, F, 9);                                                       \
        else if (d <= 12288) PB_LN1(T, F, 12);                                                     \
        else PB_LN1(T, F, LN_MAXC);                                                                \
    } while (0)
    if (dtype == 1) {
        if (out_f32) PB_LN(_Float16, true); else PB_LN(_Float16, false);
    } else {
        if (out_f32) PB_LN(__bf16, true); else PB_LN(__bf16, false);
    }
#undef PB_LN
#undef PB_LN1
#undef PB_LN2
    return hipGetLastError();
}

int lm_head_blocks(int V) { return (V + LM_BLOCK_ROWS - 1) / LM_BLOCK_ROWS; }

hipError_t launch_lm_head(int dtype, const float* z, int B, const void* E, int V, int d,
                          float* logits, float* pval, int* pidx, hipStream_t s) {
    if (B <= 0 || V <= 0) return hipSuccess;
    if (d % 8) return hipErrorInvalidValue;
    const int blocks = lm_head_blocks(V);
    for (int b0 = 0; b0 < B; b0 += 4) {
        const int nb = std::min(4, B - b0);
#define PB_LM(T, NB)                                                                           \
    PB_LAUNCH((lm_head_kernel<T, NB>), dim3(blocks), dim3(256), 0, s, z, b0,          \
                       (const T*)E, V, d, logits, pval, pidx, blocks)
        if (dtype == 1) {
            if (nb == 1) PB_LM(_Float16, 1); else if (nb == 2) PB_LM(_Float16, 2);
            else if (nb == 3) PB_LM(_Float16, 3); else PB_LM(_Float16, 4);
        } else {
            if (nb == 1) PB_LM(__bf16, 1); else if (nb == 2) PB_LM(__bf16, 2);
            else if (nb == 3) PB_LM(__bf16, 3); else PB_LM(__bf16, 4);
        }
#undef PB_LM
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_argmax(const float* pval, const int* pidx, int B, int V, int32_t* tok,
                         hipStream_t s) {
    if (B <= 0) return hipSuccess;
    PB_LAUNCH(argmax_final_kernel, dim3(B), dim3(256), 0, s, pval, pidx,
                       lm_head_blocks(V), tok);
    return hipGetLastError();
}

hipError_t launch_lora_pack(int dtype, const void* staging, size_t staging_layer_elems, int L,
                            int d, int r, uint32_t mask, int slot, int rs, int kw, void* Acat,
                            void* Bcat, hipStream_t s) {
    if (L <= 0) return hipSuccess;
    dim3 grid(L, 4, 2);
    if (dtype == 1)
        PB_LAUNCH(lora_pack_kernel<_Float16>, grid, dim3(256), 0, s,
                           (const _Float16*)staging, staging_layer_elems, d, r, mask, slot, rs, kw,
                           (_Float16*)Acat, (_Float16*)Bcat);
    else
        PB_LAUNCH(lora_pack_kernel<__bf16>, grid, dim3(256), 0, s, (const __bf16*)staging,
                           staging_layer_elems, d, r, mask, slot, rs, kw, (__bf16*)Acat,
                           (__bf16*)Bcat);
    return hipGetLastError();
}

hipError_t launch_lora_merge(int dtype, void* W, const void* Acat, const void* Bcat, int d, int kw, int rs,
                             int slot, float scale, hipStream_t s) {
    const int64_t threads = (int64_t)d * (d / 8);
    const dim3 grid((unsigned)((threads + 255) / 256));
    if (dtype == 1)
        PB_LAUNCH(lora_merge_kernel<_Float16>, grid, dim3(256), 0, s, (_Float16*)W, (const _Float16*)Acat,
                           (const _Float16*)Bcat, d, kw, rs, slot, scale);
    else
        PB_LAUNCH(lora_merge_kernel<__bf16>, grid, dim3(256), 0, s, (__bf16*)W, (const __bf16*)Acat,
                           (const __bf16*)Bcat, d, kw, rs, slot, scale);
    return hipGetLastError();
}

}  // namespace pb
