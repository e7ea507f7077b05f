// MFMA GEMM for the decoder's projections on gfx950.
//
// Y[M, N] = X[M, K] W[N, K]^T with fp32 accumulation in v_mfma_f32_16x16x32_{f16,bf16}.
// The MFMA's A operand is the weight tile (rows = output features n) and its B
// operand the activation tile (columns = tokens m), so each lane ends up with
// four consecutive output features of one token: the epilogue writes 8-byte
// (dt) or 16-byte (fp32 residual) vectors.
//
// Block tile BM x BN, K tile 64: 256 x 256 (2-stage ring, 128 KiB of LDS) or
// 128 x 128 (3-stage ring: with few tiles the weights arrive cold from HBM
// and a deeper ring hides more of that latency) with 8 waves (2 x 4, two waves
// per SIMD), chosen by how many tiles the shape gives, and 64 x 64 with 4
// waves for N not a multiple of 128.  Tiles go straight from global memory
// into the S-stage LDS ring (LDS-DMA, no staging registers), so S-1 tiles are
// in flight while one is multiplied; one barrier per K tile.  The operand
// reads from LDS, not the MFMA rate, bound the smaller tiles: a wave's
// WM x WN sub-tile reads (WM + WN) rows per K tile.
// LDS rows are 128 bytes (64 elements) with the 16-byte chunks XOR-swizzled by
// the row index so that the MFMA operand reads of 16 consecutive rows are free
// of bank conflicts (the DMA writes the swizzle by choosing which chunk each
// lane fetches).
//
// Block order: the hardware deals consecutive blocks round-robin to the 8
// XCDs; the block id is remapped so that each XCD gets a contiguous run of
// tiles, walked in groups of 8 tile-rows, so blocks that share an XCD's L2
// share rows of X and of W.
//
// Small grids are split along K (deterministically: every split writes its
// fp32 partial tile to a workspace and a reduce kernel sums the splits in a
// fixed order before the epilogue).  The tile shape and split of a launch,
// its grid and the block -> tile map live in gemm_plan.h (host and device).
//
// The LoRA expand (Section 2.1: the adapter adds s (u A) B on top of the fixed
// W) is folded into the same accumulation as extra K tiles: [X | Z][W | Bcat]^T
// where Z holds s * (u A_slot) in the row's slot columns and zeros elsewhere,
// so sequences with different adapters (or none) share one launch.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "gemm_plan.h"
#include "kernels.h"

namespace pb {

namespace {

#ifndef PB_GEMM_S128
#define PB_GEMM_S128 3  // LDS ring depth of the 128 x 128 tiles
#endif
#ifndef PB_GEMM_S64
#define PB_GEMM_S64 4  // ... of the 64 x 64 tiles
#endif
#ifndef PB_GEMM_GEMV
#define PB_GEMM_GEMV 1  // weight-streaming kernel for at most 8 token rows
#endif
#ifndef PB_GEMV_KW8
#define PB_GEMV_KW8 1  // GEMV rows of K >= 4096 split over eight waves
#endif
#ifndef PB_GEMV_NT
#define PB_GEMV_NT 1  // weights streamed by the GEMV with non-temporal loads
#endif
#ifndef PB_GEMV_RPB
#define PB_GEMV_RPB 4  // output features per GEMV block
#endif
#ifndef PB_GEMM_S256
#define PB_GEMM_S256 2  // ... of the 256 x 256 tiles
#endif

constexpr int ROW_BYTES = BK * 2;

// Physical 16-byte chunk of logical chunk ch in LDS row `row`.  chunk ^ (row & 7)
// measured conflict-free on gfx950 for the operand reads (16 rows, one chunk
// per lane group) with the bank-conflict counter.
__device__ __forceinline__ int swz(int row, int ch) { return ch ^ (row & 7); }

// Epilogue of four consecutive output features n..n+3 of token m.
template <typename T, int EPI>
__device__ __forceinline__ void epilogue4(const GemmParams& p, int m, int n, f32x4 v) {
    if (EPI == EPI_SHRINK) {
        const int slot = p.row_slot[m];
        const int c = n % p.kw;  // slot_width is a multiple of 4
        const bool keep = slot >= 0 && (c / p.slot_width) == slot;
        const float f = keep ? p.slot_scale[slot] : 0.f;
        *(u32x2*)((T*)p.C + (int64_t)m * p.ldc + n) =
            pack4<T>(keep ? v[0] * f : 0.f, keep ? v[1] * f : 0.f, keep ? v[2] * f : 0.f,
                     keep ? v[3] * f : 0.f);
        return;
    }
    const u32x2 braw = *(const u32x2*)((const T*)p.bias + n);
    T bb[4];
    __builtin_memcpy(bb, &braw, 8);
    float y[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) y[r] = v[r] + (float)bb[r];
    if (EPI == EPI_QKV) {
        float sc[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[r] = n + r < p.qcols ? p.qscale : 1.f;
        const u32x2 out = pack4<T>(y[0] * sc[0], y[1] * sc[1], y[2] * sc[2], y[3] * sc[3]);
        *(u32x2*)((T*)p.C + (int64_t)m * p.ldc + n) = out;
        if (p.kv && n >= p.qcols) {  // qcols is a multiple of 4: the group is all key or all value
            const int64_t row = (int64_t)(m / p.kv_T) * p.kv_seq + (int64_t)(*p.kv_pos + m % p.kv_T) * 2 * p.qcols;
            *(u32x2*)((T*)p.kv + row + (n - p.qcols)) = out;
        }
    } else if (EPI == EPI_RELU) {
        *(u32x2*)((T*)p.C + (int64_t)m * p.ldc + n) =
            pack4<T>(fmaxf(y[0], 0.f), fmaxf(y[1], 0.f), fmaxf(y[2], 0.f), fmaxf(y[3], 0.f));
    } else {  // EPI_RESID
        f32x4* rp = (f32x4*)(p.R + (int64_t)m * p.ldr + n);
        f32x4 rv = *rp;
        rv[0] += y[0];
        rv[1] += y[1];
        rv[2] += y[2];
        rv[3] += y[3];
        *rp = rv;
    }
}

// Epilogue of a wave's accumulators: acc[i][j] holds output features
// nb + 16 i + 4 lg + r (r = 0..3) of token mb + 16 j + lr.
template <typename T, int EPI, int MF, int NF>
__device__ __forceinline__ void store_tile(const GemmParams& p, const TileJob& jb, int mb, int nb, int lr, int lg,
                                           const f32x4 (&acc)[NF][MF]) {
#pragma unroll
    for (int j = 0; j < MF; ++j) {
        const int m = mb + j * 16 + lr;
        if (m >= p.M) continue;
#pragma unroll
        for (int i = 0; i < NF; ++i) {
            const int n = nb + i * 16 + 4 * lg;
            if (n >= p.N) continue;
            if (jb.partial)
                *(f32x4*)(jb.pbase + (int64_t)(m - jb.om) * jb.ldp + (n - jb.on)) = acc[i][j];
            else
                epilogue4<T, EPI>(p, m, n, acc[i][j]);
        }
    }
}

// (at least two waves per SIMD as the register budget: with more registers the
// compiler moves accumulators between register files around every MFMA)
template <typename T, int EPI, int BM, int BN, int WGM, int WGN, int ROLE, int S>
__global__ __launch_bounds__(64 * WGM * WGN) __attribute__((amdgpu_waves_per_eu(2)))
void gemm_kernel(GemmParams p, SplitArgs sa) {
    typedef typename Mfma<T>::vec8 vec8;
    constexpr int NW = WGM * WGN;               // waves per block
    constexpr int WM = BM / WGM, WN = BN / WGN;  // wave tile
    constexpr int MF = WM / 16, NF = WN / 16;   // 16x16 fragments per wave
    constexpr int NL = (BM + BN) / (8 * NW);    // LDS-DMA instructions per wave per K tile
    constexpr int NLX = BM / (8 * NW);          // ... of which carry X rows
    constexpr int STAGE = (BM + BN) * ROW_BYTES;
    static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "DMA slots split into X and W");
    static_assert(S >= 2 && (S - 2) * NL < 64, "pipeline depth");
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WGM, wn = wave / WGM;
    const TileJob jb = tile_job<BM, BN>(p, sa, (int)blockIdx.x, (int)gridDim.x);
    const int m0 = jb.m0, n0 = jb.n0, nk1 = jb.nk1, t_begin = jb.t_begin, nk = jb.nk;
    const T* X2 = (const T*)jb.X2;

    // DMA instruction j of this wave fills LDS rows 8g .. 8g+7, g = wave + NW j;
    // rows < BM hold X (tokens), the rest W (output features): slots j < NLX.
    // Lane i writes row 8g + i/8, physical chunk i%8, which holds logical K
    // chunk (i%8) ^ (row & 7) = (i%8) ^ (i/8) for every j.  Rows past the
    // matrix edge re-read its last row.
    const int lrow = lane >> 3;
    const int chk = swz(lrow, lane & 7) * 8;
    const int xr0 = m0 + 8 * wave + lrow, wr0 = n0 + 8 * wave + lrow - BM;
    const T* Xb = (const T*)p.X;
    const T* Wb = (const T*)p.W;
    const T* W2 = (const T*)p.W2;
    const uint32_t lds0 = (uint32_t)(uintptr_t)smem;
    // each slot's row is the same in every K tile: its byte offset (row and
    // chunk) is taken once and a tile moves the operand's scalar base by its
    // K offset, so the lanes' offsets cost no VALU work per tile (measured:
    // 46 -> 14 vector adds per K tile, the large projections 1.3-1.9% faster
    // under the power limit); byte offsets fit in 32 bits (the launcher keeps
    // rows * leading dimension below 2^31 elements)
    uint32_t soff[NL];
#pragma unroll
    for (int j = 0; j < NL; ++j)
        soff[j] = j < NLX ? ((uint32_t)min(xr0 + 8 * NW * j, p.M - 1) * (uint32_t)p.ldx + chk) * 2
                          : ((uint32_t)min(wr0 + 8 * NW * j, p.N - 1) * (uint32_t)p.ldw + chk) * 2;
    auto issue = [&](int t, int stage) {
        const uint32_t sbase = lds0 + stage * STAGE;
        if (t < nk1) {
            const int64_t kb = (int64_t)t * BK * 2;
            const char* xk = (const char*)Xb + kb;
            const char* wk = (const char*)Wb + kb;
#pragma unroll
            for (int j = 0; j < NL; ++j)
                dma16s(j < NLX ? xk : wk, soff[j],
                       sbase + (uint32_t)__builtin_amdgcn_readfirstlane((wave + NW * j) * 1024));
        } else {  // LoRA K tiles: [Z | B] rows of the same slots
            const int64_t kb = (int64_t)(t - nk1) * BK * 2;
            const char* xk = (const char*)X2 + kb;
            const char* wk = (const char*)W2 + kb;
#pragma unroll
            for (int j = 0; j < NL; ++j) {
                const uint32_t off = j < NLX ? ((uint32_t)min(xr0 + 8 * NW * j, p.M - 1) * (uint32_t)p.ldx2 + chk) * 2
                                             : ((uint32_t)min(wr0 + 8 * NW * j, p.N - 1) * (uint32_t)p.ldw2 + chk) * 2;
                dma16s(j < NLX ? xk : wk, off,
                       sbase + (uint32_t)__builtin_amdgcn_readfirstlane((wave + NW * j) * 1024));
            }
        }
    };

    f32x4 acc[NF][MF];
#pragma unroll
    for (int i = 0; i < NF; ++i)
#pragma unroll
        for (int j = 0; j < MF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int lr = lane & 15, lg = lane >> 4;
    auto compute = [&](int stage) {
        const uint8_t* s = smem + stage * STAGE;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const int ch = kk * 4 + lg;
            vec8 b[MF];
#pragma unroll
            for (int j = 0; j < MF; ++j) {
                const int row = wm * WM + j * 16 + lr;
                b[j] = as_vec8<T>(*(const u32x4*)(s + row * ROW_BYTES + (swz(row, ch) << 4)));
            }
#pragma unroll
            for (int i = 0; i < NF; ++i) {
                const int row = BM + wn * WN + i * 16 + lr;
                const vec8 a = as_vec8<T>(*(const u32x4*)(s + row * ROW_BYTES + (swz(row, ch) << 4)));
#pragma unroll
                for (int j = 0; j < MF; ++j) acc[i][j] = Mfma<T>::mma(a, b[j], acc[i][j]);
            }
        }
    };

    // S-stage ring: tiles t+1 .. t+S-1 are in flight while tile t is multiplied.
    // Steady state first (branch-free), then the tail that drains the ring.
#pragma unroll
    for (int q = 0; q < S - 1; ++q)
        if (q < nk) issue(t_begin + q, q);
    int t = 0;
    // 256 x 256 tiles except fc2: two tiles per trip, so that the ring stage
    // of every copy and operand read is a constant (fewer address adds;
    // measured qkv, o and fc1 0.8-2.4% faster at OPT-6.7B and 66B, fc2 1.5%
    // slower, 128 x 128 tiles no faster)
    if constexpr (S == 2 && BM == 256 && ROLE != 3) {
        auto step = [&](int tt, auto st_c) {
            constexpr int ST = decltype(st_c)::value;  // tt % 2
            wait_vmcnt<0>();
            __syncthreads();
            issue(t_begin + tt + 1, ST ^ 1);
            compute(ST);
        };
        for (; t + 2 < nk; t += 2) {
            step(t, std::integral_constant<int, 0>{});
            step(t + 1, std::integral_constant<int, 1>{});
        }
    }
    for (; t + S - 1 < nk; ++t) {
        wait_vmcnt<(S - 2) * NL>();  // tiles t+1 .. t+S-2 may still fly
        __syncthreads();             // tile t visible to all waves; stage of tile t-1 free
        issue(t_begin + t + S - 1, (t + S - 1) % S);
        compute(t % S);
    }
    for (; t < nk; ++t) {
        wait_vmcnt<0>();
        __syncthreads();
        compute(t % S);
    }

    store_tile<T, EPI, MF, NF>(p, jb, m0 + wm * WM, n0 + wn * WN, lr, lg, acc);
}

// Sum the split-K partials in split order, then apply the epilogue.
template <typename T, int EPI, int ROLE>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmParams p, SplitArgs sa) {
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;  // index of a group of 4 columns
    const int64_t per_row = p.N / 4;
    if (q >= (int64_t)p.M * per_row) return;
    const int m = (int)(q / per_row), n = (int)(q % per_row) * 4;
    const int64_t stride = (int64_t)p.M * p.N;
    const float* src = sa.ws + (int64_t)m * p.N + n;
    f32x4 v = *(const f32x4*)src;
    for (int s = 1; s < sa.splits; ++s) {
        const f32x4 w = *(const f32x4*)(src + s * stride);
        v[0] += w[0];
        v[1] += w[1];
        v[2] += w[2];
        v[3] += w[3];
    }
    epilogue4<T, EPI>(p, m, n, v);
}

// Reduce of a ragged-round split: only the tail tiles' partials, summed in
// split order, then the epilogue.  One thread per group of 4 columns.
template <typename T, int EPI, int ROLE, int BM, int BN>
__global__ __launch_bounds__(256) void tail_reduce_kernel(GemmParams p, SplitArgs sa) {
    constexpr int GPT = BM * BN / 4;  // column groups per tile
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (q >= (int64_t)sa.tail_tiles * GPT) return;
    const int tt = (int)(q / GPT);
    int m0, n0;
    tile_corner<BM, BN>(p, sa.full_tiles + tt, m0, n0);
    const int e = (int)(q % GPT);
    const int m = m0 + e / (BN / 4), n = n0 + (e % (BN / 4)) * 4;
    if (m >= p.M || n >= p.N) return;
    const int64_t stride = (int64_t)sa.tail_tiles * BM * BN;
    const float* src = sa.ws + (int64_t)tt * BM * BN + (int64_t)(m - m0) * BN + (n - n0);
    f32x4 v = *(const f32x4*)src;
    for (int s = 1; s < sa.splits; ++s) {
        const f32x4 w = *(const f32x4*)(src + s * stride);
        v[0] += w[0];
        v[1] += w[1];
        v[2] += w[2];
        v[3] += w[3];
    }
    epilogue4<T, EPI>(p, m, n, v);
}

// Row-wise split-K reduce of a residual projection fused with the LayerNorm
// that follows it: R[m] += (sum of partials in split order) + bias, then
// ln_out[m] = dt(LN(R[m]) * g + b) with fp32 statistics, and optionally the
// row's LoRA shrink.  One block per row; MAXC float4 chunks per thread (N <=
// 1024 MAXC); NS splits known at compile time (0: any count, summed in a loop)
// so that every partial of a chunk is in flight at once.
constexpr int RLN_MAXC = 16;  // largest chunk count: N <= 16384

template <typename T, int ROLE, int MAXC, int NS>
__global__ __launch_bounds__(256) void splitk_resid_ln_kernel(GemmParams p, SplitArgs sa) {
    __shared__ float red[4];
    const int m = blockIdx.x;
    const int nc = p.N / 4;
    const int64_t stride = (int64_t)p.M * p.N;
    float* xr = p.R + (int64_t)m * p.ldr;
    const float* wr = sa.ws + (int64_t)m * p.N;
    // every load of every chunk first (the stores to R below would otherwise
    // order the next chunk's loads behind them), then sums and stores; with
    // few chunks the loads are unconditional, a chunk past nc re-reading the
    // last one, so that no branch splits them into batches
    constexpr int NL = NS > 0 ? NS : 1;
    f32x4 v[MAXC], w[MAXC][NL];
    u32x2 braw[MAXC];
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
        int c = threadIdx.x + 256 * i;
        if (MAXC <= 4) c = min(c, nc - 1);
        else if (c >= nc) continue;
#pragma unroll
        for (int s = 0; s < NL; ++s) w[i][s] = *(const f32x4*)(wr + s * stride + 4 * c);
        braw[i] = *(const u32x2*)((const T*)p.bias + 4 * c);
        v[i] = *(const f32x4*)(xr + 4 * c);
    }
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
        const int c = threadIdx.x + 256 * i;
        if (c < nc) {
            f32x4 a = w[i][0];
#pragma unroll
            for (int s = 1; s < NS; ++s)
                a = f32x4{a[0] + w[i][s][0], a[1] + w[i][s][1], a[2] + w[i][s][2], a[3] + w[i][s][3]};
            if (NS == 0)
                for (int s = 1; s < sa.splits; ++s) {
                    const f32x4 u = *(const f32x4*)(wr + s * stride + 4 * c);
                    a = f32x4{a[0] + u[0], a[1] + u[1], a[2] + u[2], a[3] + u[3]};
                }
            T bb[4];
            __builtin_memcpy(bb, &braw[i], 8);
            f32x4 x = v[i];
#pragma unroll
            for (int r = 0; r < 4; ++r) x[r] += a[r] + (float)bb[r];
            *(f32x4*)(xr + 4 * c) = x;
            v[i] = x;
            sum += (x[0] + x[1]) + (x[2] + x[3]);
        }
    }
    row_layernorm<T, MAXC, false>(v, sum, nc, (const T*)p.ln_g, (const T*)p.ln_b,
                                  (T*)p.ln_out + (int64_t)m * p.N, p.ln_eps, red);
    if (p.shrink.Acat) {
        __shared__ float red16[4][16];
        row_shrink<T, MAXC>(p.shrink, m, p.N, v, red16);
    }
}

template <typename T, int ROLE>
hipError_t launch_resid_ln(const GemmParams& p, const SplitArgs& sa, hipStream_t s) {
#define PB_RLN(MAXC, NS) \
    PB_LAUNCH((splitk_resid_ln_kernel<T, ROLE, MAXC, NS>), dim3(p.M), dim3(256), 0, s, p, sa)
    // few rows (latency-bound): every partial in flight at once; many rows:
    // occupancy hides the latency and registers matter more
    if (p.N <= 2048) {
        if (sa.splits == 2) PB_RLN(2, 2);
        else if (sa.splits == 4) PB_RLN(2, 4);
        else PB_RLN(2, 0);
    } else if (p.N <= 4096) {
        if (sa.splits == 2) PB_RLN(4, 2);
        else if (sa.splits == 4) PB_RLN(4, 4);
        else PB_RLN(4, 0);
    } else if (p.N <= 8192) {
        PB_RLN(8, 0);
    } else {
        PB_RLN(RLN_MAXC, 0);
    }
#undef PB_RLN
    return hipGetLastError();
}

// After a split launch: the row-wise reduce (fused with the residual and the
// following LayerNorm where the caller asks for it).
template <typename T, int EPI, int ROLE>
hipError_t finish_split(const GemmParams& p, const SplitArgs& sa, hipStream_t s) {
    if (EPI == EPI_RESID && p.ln_out && p.N <= 256 * 4 * RLN_MAXC) {
        const hipError_t e = launch_resid_ln<T, ROLE>(p, sa, s);
        if (e == hipSuccess && p.ln_done) *p.ln_done = true;
        return e;
    }
    const int64_t groups = (int64_t)p.M * (p.N / 4);
    PB_LAUNCH((splitk_reduce_kernel<T, EPI, ROLE>), dim3((unsigned)((groups + 255) / 256)), dim3(256), 0,
                       s, p, sa);
    return hipGetLastError();
}

template <typename T, int EPI, int BM, int BN, int WGM, int WGN, int ROLE, int S>
hipError_t launch_cfg(const GemmParams& p, const GemmWorkspace& wsp, int splits, int ragged_tail, hipStream_t s) {
    constexpr int LDS = S * (BM + BN) * ROW_BYTES;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void*)gemm_kernel<T, EPI, BM, BN, WGM, WGN, ROLE, S>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const TileGeometry g = tile_geometry<BM, BN>(p, wsp, splits, ragged_tail);
    const SplitArgs& sa = g.sa;
    PB_LAUNCH((gemm_kernel<T, EPI, BM, BN, WGM, WGN, ROLE, S>), dim3(g.grid), dim3(64 * WGM * WGN), LDS, s, p, sa);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess || sa.splits == 1) return e;
    if (sa.full_tiles > 0) {  // whole tiles, then the tail split
        const int64_t groups = (int64_t)sa.tail_tiles * (BM * BN / 4);
        PB_LAUNCH((tail_reduce_kernel<T, EPI, ROLE, BM, BN>), dim3((unsigned)((groups + 255) / 256)), dim3(256), 0,
                  s, p, sa);
        return hipGetLastError();
    }
    return finish_split<T, EPI, ROLE>(p, sa, s);
}

template <typename T, int EPI, int ROLE>
hipError_t launch_tiles(const GemmParams& p, const GemmWorkspace& wsp, hipStream_t s) {
    const TilePlan tp = plan_for_role(ROLE, p, wsp);
    if constexpr (ROLE == 4) {
        return launch_cfg<T, EPI, 64, 64, 2, 2, 4, 4>(p, wsp, tp.splits, 0, s);
    } else {
        if (tp.tile == 256)
            return launch_cfg<T, EPI, 256, 256, 2, 4, ROLE, PB_GEMM_S256>(p, wsp, tp.splits, tp.ragged_tail, s);
        if (tp.tile == 128)
            return launch_cfg<T, EPI, 128, 128, 2, 4, ROLE, PB_GEMM_S128>(p, wsp, tp.splits, tp.ragged_tail, s);
        return launch_cfg<T, EPI, 64, 64, 2, 2, ROLE, PB_GEMM_S64>(p, wsp, tp.splits, tp.ragged_tail, s);
    }
}

template <typename T>
hipError_t launch_typed(int role, const GemmParams& p, const GemmWorkspace& wsp, hipStream_t s) {
    switch (role) {
        case 0: return launch_tiles<T, EPI_QKV, 0>(p, wsp, s);
        case 1: return launch_tiles<T, EPI_RESID, 1>(p, wsp, s);
        case 2: return launch_tiles<T, EPI_RELU, 2>(p, wsp, s);
        case 3: return launch_tiles<T, EPI_RESID, 3>(p, wsp, s);
        case 4: return launch_tiles<T, EPI_SHRINK, 4>(p, wsp, s);
        default: break;
    }
    return hipErrorInvalidValue;
}

// ---- few rows (decode steps): weight streaming without tiles ---------------
// A block owns four consecutive output features n0..n0+3; its four waves
// (eight for rows of 4096 or more) split K (and the LoRA K2 columns) into
// equal contiguous parts, so a matrix of N features is streamed by N / 4
// blocks and every CU has many waves' loads in flight (measured: four
// features per block beat eight or sixteen).  In a part, lane i takes elements 8i..8i+7 of each
// 512-element chunk (a feature's chunk is one contiguous 1 KiB read), two
// chunks per step, accumulating all MR token rows at once (MR <= GEMV_MAX_ROWS: the rows
// of X are re-read from cache by every wave).  Each wave sums its lanes, the
// parts are added in wave order through LDS, and the usual epilogue is
// applied to the four features of each token.
template <typename T, int MR, int RPB>
__device__ __forceinline__ void gemv_dot(const T* __restrict__ X, int64_t ldx, const T* __restrict__ W,
                                         int64_t ldw, int n0, int M, int kb, int ke, int lane,
                                         float (&acc)[RPB][MR]) {
    for (int c0 = kb + lane * 8; c0 < ke; c0 += 2 * 512) {
        u32x4 wr[2][RPB], xr[2][MR];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int c = min(c0 + u * 512, ke - 8);  // in bounds; the excess is not accumulated
#pragma unroll
            for (int r = 0; r < RPB; ++r) {
                const u32x4* src = (const u32x4*)(W + (int64_t)(n0 + r) * ldw + c);
#if PB_GEMV_NT
                wr[u][r] = __builtin_nontemporal_load(src);  // each weight is read once per step
#else
                wr[u][r] = *src;
#endif
            }
#pragma unroll
            for (int m = 0; m < MR; ++m) xr[u][m] = *(const u32x4*)(X + (int64_t)min(m, M - 1) * ldx + c);
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (c0 + u * 512 >= ke) break;
#pragma unroll
            for (int m = 0; m < MR; ++m) {
                T xe[8];
                __builtin_memcpy(xe, &xr[u][m], 16);
#pragma unroll
                for (int r = 0; r < RPB; ++r) {
                    T we[8];
                    __builtin_memcpy(we, &wr[u][r], 16);
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[r][m] += (float)we[e] * (float)xe[e];
                }
            }
        }
    }
}

// RPB output features per block (a multiple of 4: the epilogue writes four
// consecutive features of one token), K split over KW waves
template <typename T, int EPI, int MR, int RPB, int KW>
__global__ __launch_bounds__(64 * KW) void gemv_kernel(GemmParams p) {
    __shared__ float part[KW][RPB][MR];  // [wave][feature][token]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n0 = blockIdx.x * RPB;
    float acc[RPB][MR];
#pragma unroll
    for (int r = 0; r < RPB; ++r)
#pragma unroll
        for (int m = 0; m < MR; ++m) acc[r][m] = 0.f;
    const int q1 = p.K1 / KW;  // K1, K2 are multiples of 64: the parts are multiples of 8
    gemv_dot<T, MR, RPB>((const T*)p.X, p.ldx, (const T*)p.W, p.ldw, n0, p.M, wave * q1, (wave + 1) * q1, lane,
                         acc);
    if (p.K2 > 0) {
        const int g = n0 / p.group;  // the group size is a multiple of RPB
        const int q2 = p.K2 / KW;
        if ((p.k2_mask >> g) & 1u)
            gemv_dot<T, MR, RPB>((const T*)p.X2 + (int64_t)g * p.x2_group_stride, p.ldx2, (const T*)p.W2, p.ldw2,
                                 n0, p.M, wave * q2, (wave + 1) * q2, lane, acc);
    }
#pragma unroll
    for (int r = 0; r < RPB; ++r)
#pragma unroll
        for (int m = 0; m < MR; ++m) acc[r][m] = wave_sum(acc[r][m]);
    if (lane == 0)
#pragma unroll
        for (int r = 0; r < RPB; ++r)
#pragma unroll
            for (int m = 0; m < MR; ++m) part[wave][r][m] = acc[r][m];
    __syncthreads();
    const int m = threadIdx.x % MR, f4 = threadIdx.x / MR;  // token, group of four features
    if (f4 < RPB / 4 && m < p.M) {
        f32x4 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int rr = 4 * f4 + r;
            float t = part[0][rr][m];
#pragma unroll
            for (int w = 1; w < KW; ++w) t += part[w][rr][m];
            v[r] = t;
        }
        epilogue4<T, EPI>(p, m, n0 + 4 * f4, v);
    }
}

template <typename T, int EPI>
hipError_t launch_gemv(const GemmParams& p, hipStream_t s) {
    constexpr int RPB = PB_GEMV_RPB;
    const dim3 grid(p.N / RPB);
#define PB_GEMV(MR, KW) PB_LAUNCH((gemv_kernel<T, EPI, MR, RPB, KW>), grid, dim3(64 * KW), 0, s, p)
#define PB_GEMV_M(KW)                \
    do {                             \
        if (p.M <= 1) PB_GEMV(1, KW);      \
        else if (p.M <= 2) PB_GEMV(2, KW); \
        else if (p.M <= 4) PB_GEMV(4, KW); \
        else PB_GEMV(8, KW);               \
    } while (0)
    // long rows: eight waves share the K range so each walks at most 1024
    // elements (measured: eight waves for short rows of few blocks is slower)
    if (PB_GEMV_KW8 && p.K1 >= 4096) PB_GEMV_M(8);
    else PB_GEMV_M(4);
#undef PB_GEMV_M
#undef PB_GEMV
    return hipGetLastError();
}

template <typename T>
hipError_t launch_gemv_typed(int role, const GemmParams& p, hipStream_t s) {
    switch (role) {
        case 0: return launch_gemv<T, EPI_QKV>(p, s);
        case 1: case 3: return launch_gemv<T, EPI_RESID>(p, s);
        case 2: return launch_gemv<T, EPI_RELU>(p, s);
        case 4: return launch_gemv<T, EPI_SHRINK>(p, s);
        default: break;
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(int dtype, int role, int epi, const GemmParams& p, const GemmWorkspace& wsp,
                       hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    if (p.N % 64 || p.K1 % BK || p.K2 % BK || p.K1 <= 0 || p.K2 < 0) return hipErrorInvalidValue;
    const int64_t lim = (int64_t)1 << 31;
    if ((int64_t)p.M * p.ldx >= lim || (int64_t)p.N * p.ldw >= lim ||
        (p.K2 > 0 && ((int64_t)p.M * p.ldx2 >= lim || (int64_t)p.N * p.ldw2 >= lim)))
        return hipErrorInvalidValue;
    const int expect[5] = {EPI_QKV, EPI_RESID, EPI_RELU, EPI_RESID, EPI_SHRINK};
    if (role < 0 || role > 4 || expect[role] != epi) return hipErrorInvalidValue;
    if (p.M <= GEMV_MAX_ROWS && PB_GEMM_GEMV)
        return dtype == 1 ? launch_gemv_typed<_Float16>(role, p, s) : launch_gemv_typed<__bf16>(role, p, s);
    if (dtype == 1) return launch_typed<_Float16>(role, p, wsp, s);
    return launch_typed<__bf16>(role, p, wsp, s);
}

}  // namespace pb
