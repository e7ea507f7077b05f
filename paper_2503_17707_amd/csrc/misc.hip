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
#ifndef PB_LN_FEW_G
#define PB_LN_FEW_G 4  // ranks per shrink block of a launch with few rows
#endif
#ifndef PB_LN_AHEAD
#define PB_LN_AHEAD 1  // ... whose slot and first A rows are requested before the LayerNorm
#endif

// SHRINK: the row's LoRA shrink rides along (compiled only where it is used,
// since its registers would lower the occupancy of the plain kernel), in
// groups of G ranks; AHEAD: the slot and the block's first group of A rows
// are requested before the row's LayerNorm (launches of few rows)
template <typename T, bool OUT_F32, int MAXC, bool SHRINK, int G, bool AHEAD>
__global__ __launch_bounds__(256) void layernorm_kernel(const float* __restrict__ x,
                                                       int64_t in_mul, int64_t in_add,
                                                       const T* __restrict__ g,
                                                       const T* __restrict__ b, void* out,
                                                       int d, float eps, RowShrink sh) {
    __shared__ float red[4];
    const int row = blockIdx.x;
    const float* xr = x + ((int64_t)row * in_mul + in_add) * d;
    const int nc = d / 4;
    constexpr bool PRE = SHRINK && AHEAD && !OUT_F32;
    const int slot = PRE ? sh.row_slot[row] : -1;
    f32x4 v[MAXC];
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
        const int c = threadIdx.x + 256 * i;
        if (c < nc) v[i] = *(const f32x4*)(xr + 4 * c);
    }
    ShrinkAhead<MAXC, G> ahead;
    if (PRE) shrink_ahead<T, MAXC, G>(sh, d, slot, (int)blockIdx.y, (int)gridDim.y, ahead);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
        const int c = threadIdx.x + 256 * i;
        if (c < nc) s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
    }
    // with gridDim.y > 1 every block of the row normalizes it, block 0 writes
    // it, and the blocks share the row's LoRA shrink
    void* orow = OUT_F32 ? (void*)((float*)out + (int64_t)row * d) : (void*)((T*)out + (int64_t)row * d);
    row_layernorm<T, MAXC, OUT_F32>(v, s, nc, g, b, blockIdx.y == 0 ? orow : nullptr, eps, red);
    if (!OUT_F32 && SHRINK) {
        __shared__ float red16[4][16];
        row_shrink<T, MAXC, G>(sh, row, d, v, red16, (int)blockIdx.y, (int)gridDim.y, PRE ? &ahead : nullptr);
    }
}

// ---- LM head + argmax partials ----------------------------------------------
// logits[b, v] = z[b] . E[v] for NB sequences at once, and per block the
// (max, lowest index) of the rows it covered for each sequence, so the final
// argmax only scans one partial per block.
#ifndef PB_LM_NT
#define PB_LM_NT 1  // embedding rows read with non-temporal loads (each row is read once)
#endif

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

// The embedding is read as one stream: block b takes rows b, b + G, b + 2G, ...
// (G blocks), so at any moment the grid reads a contiguous window of rows,
// and thread t always covers the same 16-byte chunks t, t + 256, ... of a row
// (its slice of z stays in registers).  R rows are read per round; their
// per-thread partial sums are added over the block by halving exchanges and
// one LDS round; the next round's rows are requested before this round is
// reduced.  (Rows read by 8-row groups per wave, 8 consecutive rows per wave:
// 5.3 TB/s at OPT-1.3B; this order: 5.7, and 6.5 at OPT-66B.)
constexpr int LM_GRID = 512;  // 2 blocks per CU (256, 384, 640, 768, 1024 and 2048 measured slower)

// Sum over the 64 lanes of each of M (a power of two) per-lane values by
// halving exchanges in place: lane l ends with the total of value index
// l >> (6 - log2 M), the same exchanges and sums as wave_sum_multi.  The LM
// head keeps this form: its loop measured 35.1-35.5 us at OPT-1.3B against
// 37.2-37.7 with the fresh-array form, which needs fewer registers.
template <int M>
__device__ __forceinline__ float wave_sum_inplace(float (&p)[M], int lane) {
    constexpr int L = M == 1 ? 0 : M == 2 ? 1 : M == 4 ? 2 : M == 8 ? 3 : M == 16 ? 4 : 5;
    static_assert((1 << L) == M && M <= 32, "power of two up to 32");
#pragma unroll
    for (int st = 0; st < L; ++st) {
        const int D = 32 >> st;       // exchange distance
        const int n = M >> (st + 1);  // values kept
        const bool up = (lane & D) != 0;
#pragma unroll
        for (int k = 0; k < n; ++k) {
            const float send = up ? p[k] : p[n + k];
            p[k] = (up ? p[n + k] : p[k]) + __shfl_xor(send, D, 64);
        }
    }
    float a = p[0];
#pragma unroll
    for (int D = 32 >> L; D > 0; D >>= 1) a += __shfl_xor(a, D, 64);
    return a;
}

template <typename T, int NB, int CPT, int R>
__global__ __launch_bounds__(256) void lm_head_kernel(const float* __restrict__ z, int b0,
                                                     const T* __restrict__ E, int V, int d,
                                                     float* __restrict__ logits,
                                                     float* __restrict__ pval,
                                                     int* __restrict__ pidx, int nblk) {
    constexpr int M = R * NB;  // value index m = r NB + j: row r of the round, sequence j
    constexpr int SH = M == 1 ? 6 : M == 2 ? 5 : M == 4 ? 4 : M == 8 ? 3 : M == 16 ? 2 : 1;
    __shared__ float red[4][M];
    __shared__ float sv[M];
    __shared__ int si[M];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int nch = d >> 3;  // 16-byte chunks per row
    const int G = (int)gridDim.x;
    float zr[NB][CPT][8];
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = t + 256 * i;
            f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f}, bq = a;
            if (c < nch) {
                a = *(const f32x4*)(z + (int64_t)(b0 + j) * d + 8 * c);
                bq = *(const f32x4*)(z + (int64_t)(b0 + j) * d + 8 * c + 4);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                zr[j][i][e] = a[e];
                zr[j][i][4 + e] = bq[e];
            }
        }
    float best = -INFINITY;  // thread t < M: sequence t % NB over the rows it finished
    int bidx = 0x7fffffff;
    auto load = [&](u32x4 (&ev)[R][CPT], int v0) {
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int i = 0; i < CPT; ++i) {
                // rows past V and chunks past the row read an in-bounds
                // chunk (no branch around the load) and count as zeros
                const int row = v0 + G * r, c = t + 256 * i;
                const u32x4* src = (const u32x4*)(E + (int64_t)min(row, V - 1) * d + 8 * min(c, nch - 1));
#if PB_LM_NT
                const u32x4 x = __builtin_nontemporal_load(src);
#else
                const u32x4 x = *src;
#endif
                ev[r][i] = (row < V && c < nch) ? x : u32x4{0u, 0u, 0u, 0u};
            }
    };
    u32x4 ev[R][CPT], en[R][CPT];
    load(ev, (int)blockIdx.x);
    for (int v0 = (int)blockIdx.x; v0 < V; v0 += R * G) {
        load(en, v0 + R * G);
        asm volatile("" ::: "memory");  // keeps those requests ahead of this round's work
        float acc[M];
#pragma unroll
        for (int m = 0; m < M; ++m) acc[m] = 0.f;
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int i = 0; i < CPT; ++i) {
                T ea[8];
                __builtin_memcpy(ea, &ev[r][i], 16);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float w = (float)ea[e];
#pragma unroll
                    for (int j = 0; j < NB; ++j) acc[r * NB + j] += w * zr[j][i][e];
                }
            }
        const float tot = wave_sum_inplace<M>(acc, lane);
        if ((lane & ((1 << SH) - 1)) == 0) red[wave][lane >> SH] = tot;
        lds_barrier();
        if (t < M) {
            const float x = (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]);
            const int row = v0 + G * (t / NB);
            if (row < V) {
                logits[(int64_t)(b0 + t % NB) * V + row] = x;
                if (better(x, row, best, bidx)) {
                    best = x;
                    bidx = row;
                }
            }
        }
        lds_barrier();  // red is written again next round
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int i = 0; i < CPT; ++i) ev[r][i] = en[r][i];
    }
    if (t < M) {
        sv[t] = best;
        si[t] = bidx;
    }
    lds_barrier();
    if (t < NB) {
        float bb = sv[t];
        int ii = si[t];
        for (int r = 1; r < R; ++r)
            if (better(sv[r * NB + t], si[r * NB + t], bb, ii)) {
                bb = sv[r * NB + t];
                ii = si[r * NB + t];
            }
        pval[(int64_t)(b0 + t) * nblk + blockIdx.x] = bb;
        pidx[(int64_t)(b0 + t) * nblk + blockIdx.x] = ii;
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
    // a few rows (decode steps): the row's shrink groups of PB_LN_FEW_G ranks
    // go to blocks of their own, so that the A reads spread over several CUs
    // (many rows: groups of 16, one block per row)
    const bool few = sh.Acat && rows <= 8;
    int slices = 1;
    if (few) slices = std::max(1, __builtin_popcount(sh.mask & 7u) * ((sh.rs + PB_LN_FEW_G - 1) / PB_LN_FEW_G));
#define PB_LN2(T, F, C, SH, G, AH)                                                                 \
    PB_LAUNCH((layernorm_kernel<T, F, C, SH, G, AH>), dim3(rows, slices), dim3(256), 0, s, x, in_mul, \
              in_add, (const T*)g, (const T*)b, out, d, eps, sh)
#define PB_LN1(T, F, C)                                                                            \
    do {                                                                                           \
        if (!F && sh.Acat) {                                                                       \
            if (few) PB_LN2(T, false, C, true, PB_LN_FEW_G, PB_LN_AHEAD);                          \
            else PB_LN2(T, false, C, true, 16, false);                                             \
        } else {                                                                                   \
            PB_LN2(T, F, C, false, 16, false);                                                     \
        }                                                                                          \
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

int lm_head_blocks(int V) { return std::max(1, std::min(LM_GRID, V)); }

template <typename T, int CPT, int R, int NBMAX>
void lm_head_launch(int nb, const float* z, int b0, const void* E, int V, int d, float* logits,
                    float* pval, int* pidx, int blocks, hipStream_t s) {
#define PB_LM(NB)                                                                                \
    PB_LAUNCH((lm_head_kernel<T, NB, CPT, R>), dim3(blocks), dim3(256), 0, s, z, b0, (const T*)E, V, d, \
              logits, pval, pidx, blocks)
    if (nb == 1) {
        PB_LM(1);
    } else if constexpr (NBMAX >= 2) {
        if (nb == 2) PB_LM(2);
        else if constexpr (NBMAX >= 4) PB_LM(4);
    }
#undef PB_LM
}

hipError_t launch_lm_head(int dtype, const float* z, int B, const void* E, int V, int d,
                          float* logits, float* pval, int* pidx, hipStream_t s) {
    if (B <= 0 || V <= 0) return hipSuccess;
    if (d % 8 || d > 8 * 256 * 8) return hipErrorInvalidValue;
    const int blocks = lm_head_blocks(V);
    const int cpt = (d / 8 + 255) / 256;  // 16-byte chunks per thread per row
    // sequences per launch (a power of two): their z slices stay in registers
    const int nbmax = cpt <= 2 ? 4 : cpt <= 5 ? 2 : 1;
    for (int b0 = 0; b0 < B;) {
        int nb = 1;
        while (nb * 2 <= std::min(nbmax, B - b0)) nb *= 2;
        if (dtype == 1) {
            if (cpt == 1) lm_head_launch<_Float16, 1, 8, 4>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
            else if (cpt == 2) lm_head_launch<_Float16, 2, 4, 4>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
            else if (cpt == 3) lm_head_launch<_Float16, 3, 2, 2>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
            else if (cpt <= 5) lm_head_launch<_Float16, 5, 2, 2>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
            else lm_head_launch<_Float16, 8, 1, 1>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
        } else {
            if (cpt == 1) lm_head_launch<__bf16, 1, 8, 4>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
            else if (cpt == 2) lm_head_launch<__bf16, 2, 4, 4>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
            else if (cpt == 3) lm_head_launch<__bf16, 3, 2, 2>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
            else if (cpt <= 5) lm_head_launch<__bf16, 5, 2, 2>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
            else lm_head_launch<__bf16, 8, 1, 1>(nb, z, b0, E, V, d, logits, pval, pidx, blocks, s);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        b0 += nb;
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
