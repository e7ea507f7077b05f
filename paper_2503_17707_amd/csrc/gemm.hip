// MFMA GEMM for the decoder's projections on gfx950.
//
// Y[M, N] = X[M, K] W[N, K]^T with fp32 accumulation in v_mfma_f32_16x16x32_{f16,bf16}.
// The MFMA's A operand is the weight tile (rows = output features n) and its B
// operand the activation tile (columns = tokens m), so each lane ends up with
// four consecutive output features of one token: the epilogue writes 8-byte
// (dt) or 16-byte (fp32 residual) vectors.
//
// Block: 256 threads = 4 waves in a 2 x 2 grid; block tile BM x BN, K tile 64.
// Tiles go global -> registers -> LDS (double buffered, one barrier per K
// tile); the loads of tile t+1 are in flight while tile t is multiplied.  LDS
// rows are 128 bytes (64 elements) with the 16-byte chunks XOR-swizzled so
// that the MFMA operand reads of 16 consecutive rows hit distinct banks.
//
// The LoRA expand (Section 2.1: the adapter adds s (u A) B on top of the fixed
// W) is folded into the same accumulation as extra K tiles: [X | Z][W | Bcat]^T
// where Z holds s * (u A_slot) in the row's slot columns and zeros elsewhere,
// so sequences with different adapters (or none) share one launch.
#include "common.h"
#include "kernels.h"

namespace pb {

namespace {

constexpr int BK = 64;
constexpr int ROW_BYTES = BK * 2;

__device__ __forceinline__ int swz(int row, int ch) {
    return ch ^ ((row & 7) ^ ((row >> 3) & 1));
}

template <typename T, int EPI, int BM, int BN, int ROLE>
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p) {
    typedef typename Mfma<T>::vec8 vec8;
    constexpr int WM = BM / 2, WN = BN / 2;     // wave tile
    constexpr int MF = WM / 16, NF = WN / 16;   // 16x16 fragments per wave
    constexpr int XL = BM * 8 / 256, WL = BN * 8 / 256;  // 16-byte loads per thread
    constexpr int STAGE = (BM + BN) * ROW_BYTES;
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int tiles_m = (p.M + BM - 1) / BM;
    const int tm = blockIdx.x % tiles_m, tn = blockIdx.x / tiles_m;
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
    const int nk = nk1 + nk2;

    // per-thread load coordinates (row, 16-byte chunk) of the X and W tiles
    int64_t xoff[XL], woff[WL], x2off[XL], w2off[WL];
    int xs[XL], ws[WL];
#pragma unroll
    for (int i = 0; i < XL; ++i) {
        const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
        const int m = min(m0 + row, p.M - 1);
        xoff[i] = (int64_t)m * p.ldx + ch * 8;
        x2off[i] = (int64_t)m * p.ldx2 + ch * 8;
        xs[i] = row * ROW_BYTES + (swz(row, ch) << 4);
    }
#pragma unroll
    for (int i = 0; i < WL; ++i) {
        const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
        const int n = min(n0 + row, p.N - 1);
        woff[i] = (int64_t)n * p.ldw + ch * 8;
        w2off[i] = (int64_t)n * p.ldw2 + ch * 8;
        ws[i] = BM * ROW_BYTES + row * ROW_BYTES + (swz(row, ch) << 4);
    }

    u32x4 rx[XL], rw[WL];
    auto load = [&](int t) {
        if (t < nk1) {
            const int64_t k = (int64_t)t * BK;
#pragma unroll
            for (int i = 0; i < XL; ++i) rx[i] = *(const u32x4*)(X + xoff[i] + k);
#pragma unroll
            for (int i = 0; i < WL; ++i) rw[i] = *(const u32x4*)(W + woff[i] + k);
        } else {
            const int64_t k = (int64_t)(t - nk1) * BK;
#pragma unroll
            for (int i = 0; i < XL; ++i) rx[i] = *(const u32x4*)(X2 + x2off[i] + k);
#pragma unroll
            for (int i = 0; i < WL; ++i) rw[i] = *(const u32x4*)(W2 + w2off[i] + k);
        }
    };
    auto store = [&](int buf) {
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

    // operand read offsets inside a stage
    const int lr = lane & 15, lg = lane >> 4;
    int aoff[2][NF], boff[2][MF];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        const int ch = kk * 4 + lg;
#pragma unroll
        for (int i = 0; i < NF; ++i) {
            const int row = wn * WN + i * 16 + lr;
            aoff[kk][i] = BM * ROW_BYTES + row * ROW_BYTES + (swz(row, ch) << 4);
        }
#pragma unroll
        for (int j = 0; j < MF; ++j) {
            const int row = wm * WM + j * 16 + lr;
            boff[kk][j] = row * ROW_BYTES + (swz(row, ch) << 4);
        }
    }

    if (nk > 0) {
        load(0);
        store(0);
    }
    __syncthreads();
    for (int t = 0; t < nk; ++t) {
        if (t + 1 < nk) load(t + 1);
        const uint8_t* s = smem + (t & 1) * STAGE;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            vec8 a[NF], b[MF];
#pragma unroll
            for (int i = 0; i < NF; ++i) a[i] = as_vec8<T>(*(const u32x4*)(s + aoff[kk][i]));
#pragma unroll
            for (int j = 0; j < MF; ++j) b[j] = as_vec8<T>(*(const u32x4*)(s + boff[kk][j]));
#pragma unroll
            for (int i = 0; i < NF; ++i)
#pragma unroll
                for (int j = 0; j < MF; ++j) acc[i][j] = Mfma<T>::mma(a[i], b[j], acc[i][j]);
        }
        if (t + 1 < nk) store((t + 1) & 1);
        __syncthreads();
    }

    // epilogue: lane holds n = nb + 4*lg + r (r = 0..3) of token m
#pragma unroll
    for (int j = 0; j < MF; ++j) {
        const int m = m0 + wm * WM + j * 16 + lr;
        if (m >= p.M) continue;
        int slot = -1;
        float sscale = 0.f;
        if (EPI == EPI_SHRINK) {
            slot = p.row_slot[m];
            if (slot >= 0) sscale = p.slot_scale[slot];
        }
#pragma unroll
        for (int i = 0; i < NF; ++i) {
            const int n = n0 + wn * WN + i * 16 + 4 * lg;
            if (n >= p.N) continue;
            f32x4 v = acc[i][j];
            if (EPI == EPI_SHRINK) {
                const int c = n % p.kw;  // slot_width is a multiple of 4
                const bool keep = slot >= 0 && (c / p.slot_width) == slot;
                const float f = keep ? sscale : 0.f;
                u32x2 o = pack4<T>(keep ? v[0] * f : 0.f, keep ? v[1] * f : 0.f,
                                   keep ? v[2] * f : 0.f, keep ? v[3] * f : 0.f);
                *(u32x2*)((T*)p.C + (int64_t)m * p.ldc + n) = o;
            } else {
                const u32x2 braw = *(const u32x2*)((const T*)p.bias + n);
                T bb[4];
                __builtin_memcpy(bb, &braw, 8);
                float y[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) y[r] = v[r] + (float)bb[r];
                if (EPI == EPI_QKV) {
                    const float sc = n < p.qcols ? p.qscale : 1.f;
                    *(u32x2*)((T*)p.C + (int64_t)m * p.ldc + n) =
                        pack4<T>(y[0] * sc, y[1] * sc, y[2] * sc, y[3] * sc);
                } else if (EPI == EPI_RELU) {
                    *(u32x2*)((T*)p.C + (int64_t)m * p.ldc + n) =
                        pack4<T>(fmaxf(y[0], 0.f), fmaxf(y[1], 0.f), fmaxf(y[2], 0.f),
                                 fmaxf(y[3], 0.f));
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
        }
    }
}

template <typename T, int EPI, int BM, int BN, int ROLE>
hipError_t launch_cfg(const GemmParams& p, hipStream_t s) {
    const int tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
    hipLaunchKernelGGL((gemm_kernel<T, EPI, BM, BN, ROLE>), dim3(tiles), dim3(256), 0, s, p);
    return hipGetLastError();
}

template <typename T, int EPI, int ROLE>
hipError_t launch_tiles(const GemmParams& p, hipStream_t s) {
    // 128 x 128 tiles when they alone give every CU work; 64 x 64 otherwise.
    const long big = (long)((p.M + 127) / 128) * ((p.N + 127) / 128);
    if (big >= 256) return launch_cfg<T, EPI, 128, 128, ROLE>(p, s);
    return launch_cfg<T, EPI, 64, 64, ROLE>(p, s);
}

template <typename T>
hipError_t launch_typed(int role, int epi, const GemmParams& p, hipStream_t s) {
    switch (role) {
        case 0: return launch_tiles<T, EPI_QKV, 0>(p, s);
        case 1: return launch_tiles<T, EPI_RESID, 1>(p, s);
        case 2: return launch_tiles<T, EPI_RELU, 2>(p, s);
        case 3: return launch_tiles<T, EPI_RESID, 3>(p, s);
        case 4: return launch_tiles<T, EPI_SHRINK, 4>(p, s);
        default: break;
    }
    (void)epi;
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(int dtype, int role, int epi, const GemmParams& p, hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    if (p.N % 64 || p.K1 % BK || p.K2 % BK || p.K1 < 0 || p.K2 < 0) return hipErrorInvalidValue;
    const int expect[5] = {EPI_QKV, EPI_RESID, EPI_RELU, EPI_RESID, EPI_SHRINK};
    if (role < 0 || role > 4 || expect[role] != epi) return hipErrorInvalidValue;
    if (dtype == 1) return launch_typed<_Float16>(role, epi, p, s);
    return launch_typed<__bf16>(role, epi, p, s);
}

}  // namespace pb
