// MFMA GEMM for the decoder's projections on gfx950.
//
// Y[M, N] = X[M, K] W[N, K]^T with fp32 accumulation in v_mfma_f32_16x16x32_{f16,bf16}.
// The MFMA's A operand is the weight tile (rows = output features n) and its B
// operand the activation tile (columns = tokens m), so each lane ends up with
// four consecutive output features of one token: the epilogue writes 8-byte
// (dt) or 16-byte (fp32 residual) vectors.
//
// Block: 256 threads = 4 waves in a 2 x 2 grid; block tile BM x BN (128 x 128,
// or 64 x 64 for the LoRA shrink and for N not a multiple of 128), K tile 64.
// Tiles go global -> registers -> LDS; one or two register sets keep the
// loads of tiles t+1 (and t+2) in flight while tile t is multiplied from LDS
// (two LDS stages, one barrier per K tile).  LDS rows are 128 bytes (64 elements) with
// the 16-byte chunks XOR-swizzled so that the MFMA operand reads of 16
// consecutive rows hit distinct banks.
//
// Block order: the hardware deals consecutive blocks round-robin to the 8
// XCDs; the block id is remapped so that each XCD gets a contiguous run of
// tiles, walked in groups of 8 tile-rows, so blocks that share an XCD's L2
// share rows of X and of W.
//
// Small grids are split along K (deterministically: every split writes its
// fp32 partial tile to a workspace and a reduce kernel sums the splits in a
// fixed order before the epilogue).
//
// The LoRA expand (Section 2.1: the adapter adds s (u A) B on top of the fixed
// W) is folded into the same accumulation as extra K tiles: [X | Z][W | Bcat]^T
// where Z holds s * (u A_slot) in the row's slot columns and zeros elsewhere,
// so sequences with different adapters (or none) share one launch.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace pb {

namespace {

#ifndef PB_GEMM_PF128
#define PB_GEMM_PF128 1  // prefetch depth of the 128 x 128 tiles
#endif
#ifndef PB_GEMM_MIN_KT
#define PB_GEMM_MIN_KT 8  // fewest K tiles a split-K block gets
#endif

constexpr int BK = 64;
constexpr int ROW_BYTES = BK * 2;
constexpr int GROUP_M = 8;

__device__ __forceinline__ int swz(int row, int ch) {
    return ch ^ ((row & 7) ^ ((row >> 3) & 1));
}

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
        const float sc = n < p.qcols ? p.qscale : 1.f;
        *(u32x2*)((T*)p.C + (int64_t)m * p.ldc + n) = pack4<T>(y[0] * sc, y[1] * sc, y[2] * sc, y[3] * sc);
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

struct SplitArgs {
    int splits;     // number of K splits (1 = none)
    int kt_split;   // K tiles per split (the LoRA tiles go to the last split)
    float* ws;      // [splits][M][N] fp32 partials when splits > 1
};

template <typename T, int EPI, int BM, int BN, int ROLE, int PF>
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p, SplitArgs sa) {
    typedef typename Mfma<T>::vec8 vec8;
    constexpr int WM = BM / 2, WN = BN / 2;     // wave tile
    constexpr int MF = WM / 16, NF = WN / 16;   // 16x16 fragments per wave
    constexpr int XL = BM * 8 / 256, WL = BN * 8 / 256;  // 16-byte loads per thread
    constexpr int STAGE = (BM + BN) * ROW_BYTES;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int tiles_m = (p.M + BM - 1) / BM;
    const int tiles_n = (p.N + BN - 1) / BN;
    const int tiles = tiles_m * tiles_n;

    // XCD-contiguous block order, then split, then grouped tile order
    int bid = blockIdx.x;
    const int nblk = gridDim.x;
    if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
    const int tile = bid % tiles, split = bid / tiles;
    const int per_group = GROUP_M * tiles_n;
    const int gid = tile / per_group;
    const int first_m = gid * GROUP_M;
    const int gsize = min(tiles_m - first_m, GROUP_M);
    const int tm = first_m + (tile % per_group) % gsize;
    const int tn = (tile % per_group) / gsize;
    const int m0 = tm * BM, n0 = tn * BN;

    const T* X = (const T*)p.X;
    const T* W = (const T*)p.W;
    const int nk1 = p.K1 / BK;
    int nk2 = 0;
    const T* X2 = nullptr;
    if (p.K2 > 0) {
        const int g = n0 / p.group;
        if ((p.k2_mask >> g) & 1u) {
            nk2 = p.K2 / BK;
            X2 = (const T*)p.X2 + (int64_t)g * p.x2_group_stride;
        }
    }
    const T* W2 = (const T*)p.W2;
    // K-tile range of this split
    const int t_begin = split * sa.kt_split;
    const int t_end = (split == sa.splits - 1) ? nk1 + nk2 : min(nk1, t_begin + sa.kt_split);
    const int nk = t_end - t_begin;

    // per-thread load coordinates (row, 16-byte chunk) of the X and W tiles;
    // element offsets fit in 31 bits (checked by the launcher)
    int xoff[XL], woff[WL], xs[XL], ws[WL];
#pragma unroll
    for (int i = 0; i < XL; ++i) {
        const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
        const int m = min(m0 + row, p.M - 1);
        xoff[i] = m * (int)p.ldx + ch * 8;
        xs[i] = row * ROW_BYTES + (swz(row, ch) << 4);
    }
#pragma unroll
    for (int i = 0; i < WL; ++i) {
        const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
        const int n = min(n0 + row, p.N - 1);
        woff[i] = n * (int)p.ldw + ch * 8;
        ws[i] = BM * ROW_BYTES + row * ROW_BYTES + (swz(row, ch) << 4);
    }

    u32x4 rx0[XL], rw0[WL], rx1[XL], rw1[WL];
    auto load = [&](int t, u32x4 (&rx)[XL], u32x4 (&rw)[WL]) {
        if (t < nk1) {
            const int k = t * BK;
#pragma unroll
            for (int i = 0; i < XL; ++i) rx[i] = *(const u32x4*)(X + xoff[i] + k);
#pragma unroll
            for (int i = 0; i < WL; ++i) rw[i] = *(const u32x4*)(W + woff[i] + k);
        } else {  // LoRA expand tiles
            const int k = (t - nk1) * BK;
#pragma unroll
            for (int i = 0; i < XL; ++i) {
                const int c = tid + 256 * i;
                const int m = min(m0 + (c >> 3), p.M - 1);
                rx[i] = *(const u32x4*)(X2 + m * (int)p.ldx2 + (c & 7) * 8 + k);
            }
#pragma unroll
            for (int i = 0; i < WL; ++i) {
                const int c = tid + 256 * i;
                const int n = min(n0 + (c >> 3), p.N - 1);
                rw[i] = *(const u32x4*)(W2 + n * (int)p.ldw2 + (c & 7) * 8 + k);
            }
        }
    };
    auto store = [&](int buf, const u32x4 (&rx)[XL], const u32x4 (&rw)[WL]) {
        uint8_t* s = smem + buf * STAGE;
#pragma unroll
        for (int i = 0; i < XL; ++i) *(u32x4*)(s + xs[i]) = rx[i];
#pragma unroll
        for (int i = 0; i < WL; ++i) *(u32x4*)(s + ws[i]) = rw[i];
    };

    f32x4 acc[NF][MF];
#pragma unroll
    for (int i = 0; i < NF; ++i)
#pragma unroll
        for (int j = 0; j < MF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int lr = lane & 15, lg = lane >> 4;
    // operand read offsets inside a stage, for k step kk (0/1) of the 64-wide tile
    auto aoff = [&](int kk, int i) {
        const int row = wn * WN + i * 16 + lr, ch = kk * 4 + lg;
        return BM * ROW_BYTES + row * ROW_BYTES + (swz(row, ch) << 4);
    };
    auto boff = [&](int kk, int j) {
        const int row = wm * WM + j * 16 + lr, ch = kk * 4 + lg;
        return row * ROW_BYTES + (swz(row, ch) << 4);
    };
    auto compute = [&](int buf) {
        const uint8_t* s = smem + buf * STAGE;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            vec8 b[MF];
#pragma unroll
            for (int j = 0; j < MF; ++j) b[j] = as_vec8<T>(*(const u32x4*)(s + boff(kk, j)));
#pragma unroll
            for (int i = 0; i < NF; ++i) {
                const vec8 a = as_vec8<T>(*(const u32x4*)(s + aoff(kk, i)));
#pragma unroll
                for (int j = 0; j < MF; ++j) acc[i][j] = Mfma<T>::mma(a, b[j], acc[i][j]);
            }
        }
    };

    if constexpr (PF == 1) {
        // tile t+1 in registers while tile t is multiplied
        if (nk > 0) {
            load(t_begin, rx0, rw0);
            store(0, rx0, rw0);
        }
        __syncthreads();
        for (int t = 0; t < nk; ++t) {
            if (t + 1 < nk) load(t_begin + t + 1, rx0, rw0);
            compute(t & 1);
            if (t + 1 < nk) store((t + 1) & 1, rx0, rw0);
            __syncthreads();
        }
    } else {
        // tiles t+1 and t+2 in registers while tile t is multiplied
        if (nk > 0) {
            load(t_begin, rx0, rw0);
            if (nk > 1) load(t_begin + 1, rx1, rw1);
            store(0, rx0, rw0);
            if (nk > 2) load(t_begin + 2, rx0, rw0);
        }
        __syncthreads();
        for (int t = 0; t < nk; t += 2) {
            // even step: compute stage 0; set 1 holds tile t+1, set 0 tile t+2
            compute(0);
            if (t + 1 < nk) store(1, rx1, rw1);
            if (t + 3 < nk) load(t_begin + t + 3, rx1, rw1);
            __syncthreads();
            if (t + 1 >= nk) break;
            // odd step: compute stage 1; set 0 holds tile t+2, set 1 tile t+3
            compute(1);
            if (t + 2 < nk) store(0, rx0, rw0);
            if (t + 4 < nk) load(t_begin + t + 4, rx0, rw0);
            __syncthreads();
        }
    }

    // epilogue: lane holds n = nb + 4*lg + r (r = 0..3) of token m
#pragma unroll
    for (int j = 0; j < MF; ++j) {
        const int m = m0 + wm * WM + j * 16 + lr;
        if (m >= p.M) continue;
#pragma unroll
        for (int i = 0; i < NF; ++i) {
            const int n = n0 + wn * WN + i * 16 + 4 * lg;
            if (n >= p.N) continue;
            if (sa.splits > 1)
                *(f32x4*)(sa.ws + ((int64_t)split * p.M + m) * p.N + n) = acc[i][j];
            else
                epilogue4<T, EPI>(p, m, n, acc[i][j]);
        }
    }
}

// Sum the split-K partials in split order, then apply the epilogue.
template <typename T, int EPI>
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

template <typename T, int EPI, int BM, int BN, int ROLE, int PF>
hipError_t launch_cfg(const GemmParams& p, const GemmWorkspace& wsp, hipStream_t s) {
    constexpr int LDS = 2 * (BM + BN) * ROW_BYTES;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void*)gemm_kernel<T, EPI, BM, BN, ROLE, PF>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
    const int nk1 = p.K1 / BK;
    // split K when the tiles alone leave CUs idle, keeping >= PB_GEMM_MIN_KT
    // K tiles per split
    int splits = 1;
    if (tiles < 256 && wsp.ws && wsp.bytes > 0) {
        splits = std::min((512 + tiles - 1) / tiles, nk1 / PB_GEMM_MIN_KT);
        const int64_t per_split = (int64_t)p.M * p.N * 4;
        splits = (int)std::min<int64_t>(splits, (int64_t)(wsp.bytes / per_split));
        if (splits < 1) splits = 1;
    }
    SplitArgs sa;
    sa.kt_split = (nk1 + splits - 1) / splits;
    // splits 0..S-2 take kt_split base tiles each, the last one the rest (and
    // the LoRA tiles); S = ceil(nk1 / kt_split) leaves no split empty
    sa.splits = (nk1 + sa.kt_split - 1) / sa.kt_split;
    sa.ws = (float*)wsp.ws;
    hipLaunchKernelGGL((gemm_kernel<T, EPI, BM, BN, ROLE, PF>), dim3(tiles * sa.splits), dim3(256), LDS, s,
                       p, sa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || sa.splits == 1) return e;
    const int64_t groups = (int64_t)p.M * (p.N / 4);
    hipLaunchKernelGGL((splitk_reduce_kernel<T, EPI>), dim3((unsigned)((groups + 255) / 256)), dim3(256), 0,
                       s, p, sa);
    return hipGetLastError();
}

template <typename T, int EPI, int ROLE>
hipError_t launch_tiles(const GemmParams& p, const GemmWorkspace& wsp, hipStream_t s) {
    if (p.N % 128 == 0) return launch_cfg<T, EPI, 128, 128, ROLE, PB_GEMM_PF128>(p, wsp, s);
    return launch_cfg<T, EPI, 64, 64, ROLE, 2>(p, wsp, s);
}

template <typename T>
hipError_t launch_typed(int role, const GemmParams& p, const GemmWorkspace& wsp, hipStream_t s) {
    switch (role) {
        case 0: return launch_tiles<T, EPI_QKV, 0>(p, wsp, s);
        case 1: return launch_tiles<T, EPI_RESID, 1>(p, wsp, s);
        case 2: return launch_tiles<T, EPI_RELU, 2>(p, wsp, s);
        case 3: return launch_tiles<T, EPI_RESID, 3>(p, wsp, s);
        case 4: return launch_cfg<T, EPI_SHRINK, 64, 64, 4, 2>(p, wsp, s);
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
    if (dtype == 1) return launch_typed<_Float16>(role, p, wsp, s);
    return launch_typed<__bf16>(role, p, wsp, s);
}

}  // namespace pb
