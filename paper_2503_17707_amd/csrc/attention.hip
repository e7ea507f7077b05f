// Causal self-attention of the prefill (Section 2.1: every layer relates all
// prompt tokens through self-attention; a prefill is causal, token j sees
// tokens 0..j), flash-style: the T x T score matrix is never stored.
//
// Block = 4 waves of one (sequence, head); each wave owns 16 or 32 queries.
// Key/value tiles of 64 rows arrive row-major in a two-stage LDS ring by
// LDS-DMA (the next tile loads while this one is used) and are consumed with
// v_mfma_f32_16x16x32_{f16,bf16}:
//
//   S^T[key, query] = K Q^T      A operand = K rows, B operand = the wave's Q
//                                 (held in registers for the whole kernel)
//   O^T[c, query]  += V^T P^T    A operand = V^T rows, B operand = P^T
//
// With the transposed products every lane holds scores and outputs of one
// query (lane % 16), so the online softmax (running max m, running sum l, in
// fp32) needs only cross-lane reductions over the 4 lane groups and no
// transposition of P: the 8 keys a lane contributes to one P^T operand are the
// 8 scores it already holds.  The V^T operand is read from the row-major V
// tile with transposing LDS reads (ds_read_b64_tr_b16) in the same key order.
//
// The max and sum over a query's four lane groups use v_permlane16/32_swap
// (VALU, no LDS round trip).  Blocks run heaviest-first over all (sequence,
// head) pairs (the last query block of a pair sees the most keys).  When
// query blocks are few (a short prompt), KS = 2 wave groups of 4 share a
// block's queries and take alternating key tiles; the two online-softmax
// states are merged through LDS at the end, halving the longest block's key
// loop and putting two waves on each SIMD.
#include "common.h"
#include "kernels.h"

namespace pb {

namespace {

#ifndef PB_ATTN_QW32
#define PB_ATTN_QW32 1  // allow 32 queries per wave
#endif
#ifndef PB_ATTN_KS2
#define PB_ATTN_KS2 1  // allow two wave groups splitting the keys
#endif
#ifndef PB_ATTN_MFMA_SUM
#define PB_ATTN_MFMA_SUM 1  // softmax row sums by the matrix unit (a tile of ones in P V)
#endif
#ifndef PB_ATTN_KSWZ16
#define PB_ATTN_KSWZ16 1  // K tiles of head_dim 128 permuted over all 16 chunks
#endif
#ifndef PB_ATTN_PERMLANE
#define PB_ATTN_PERMLANE 1  // reductions over the 4 lane groups with permlane swaps
#endif

constexpr float LOG2E = 1.4426950408889634f;

// two 1.0 values of dt packed in 32 bits
template <typename T> __device__ constexpr uint32_t ONE2();
template <> __device__ constexpr uint32_t ONE2<_Float16>() { return 0x3C003C00u; }
template <> __device__ constexpr uint32_t ONE2<__bf16>() { return 0x3F803F80u; }
constexpr int BKV = 64;  // keys per tile

// 16-byte chunk permutations of a K or V tile row (key = row): K is read as
// 16 consecutive rows at one chunk, V by transposing 8-byte reads of four
// consecutive rows at two neighbouring chunks.
template <int HD>
__device__ __forceinline__ int kswz(int row, int ch) {
    // a read of 16 consecutive rows at one chunk hits 16 distinct 16-byte
    // positions of the 256-byte bank window: with 128-byte rows (row & 7) and
    // the row parity do it, with 256-byte rows the permutation needs (row & 15)
    if (HD == 128 && PB_ATTN_KSWZ16) return ch ^ (row & 15);
    return ch ^ (row & 7);
}
template <int HD>
__device__ __forceinline__ int vswz(int row, int ch) {
    // rows 4 g + j (j = 0..3) of one transposing read land in distinct banks
    // by (row & 3); bit 2 of the row moves rows 4..7 off the banks of rows
    // 0..3 (to the other half of a 256-byte row, or to the other chunk pairs
    // of a 128-byte one): half the bank conflicts of (row & 3) alone, measured
    if (HD == 128) return ch ^ ((row & 3) << 1) ^ (((row >> 2) & 1) << 3);
    return ch ^ (((row & 3) ^ ((row >> 2) & 1)) << 1);
}

// Transposing LDS read (ds_read_b64_tr_b16): within each group of 16 lanes,
// lane i receives element i % 4 of the 8-byte segments addressed by lanes
// 4 j + i / 4, j = 0..3 (layout checked on gfx950 with an in-bounds probe).
template <typename T>
__device__ __forceinline__ u32x2 read_tr16(const uint8_t* p) {
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(p));
    return __builtin_bit_cast(u32x2, v);
}

// max and sum over lanes l, l ^ 16, l ^ 32, l ^ 48 (the four 16-lane groups),
// identical in all four lanes: v_permlane16_swap of a register with itself
// hands every lane the value of the same lane position in the paired 16-lane
// row (rows 0 <-> 1, 2 <-> 3), v_permlane32_swap that of the other 32-lane
// half (layout checked on gfx950 with an in-bounds probe); plain VALU
// instructions, no LDS round trip
__device__ __forceinline__ float group4_max(float v) {
#if PB_ATTN_PERMLANE
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
#else
    v = fmaxf(v, __shfl_xor(v, 16, 64));
    return fmaxf(v, __shfl_xor(v, 32, 64));
#endif
}

__device__ __forceinline__ float group4_sum(float v) {
#if PB_ATTN_PERMLANE
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
#else
    v += __shfl_xor(v, 16, 64);
    return v + __shfl_xor(v, 32, 64);
#endif
}

template <typename T, int HD, int QW, int KS, int NQW, int S>
__global__ __launch_bounds__(64 * NQW * KS) __attribute__((amdgpu_waves_per_eu(QW == 32 || KS == 2 || NQW == 8 ? 2 : 1)))
void attention_kernel(const T* __restrict__ qkv, const T* __restrict__ kvsrc, int64_t kv_ld, int64_t kv_seq,
                      T* __restrict__ out, int T_len, int H, int B) {
    typedef typename Mfma<T>::vec8 vec8;
    constexpr int NW = NQW * KS;       // waves per block
    constexpr int BQ = NQW * QW;       // queries per block (NQW waves per group)
    constexpr int NQG = QW / 16;       // 16-query groups per wave
    constexpr int CS = HD / 32;        // 32-wide k steps over head_dim
    constexpr int CT = HD / 16;        // 16-row tiles of O^T
    constexpr int RB = HD * 2;         // bytes per K/V row
    constexpr int CPR = RB / 16;       // 16-byte chunks per row
    constexpr int TILE = BKV * RB;     // bytes per K or V tile
    constexpr int GSTAGE = 2 * TILE;   // one key tile: K then V
    constexpr int STAGE = KS * GSTAGE; // one key tile per wave group
    constexpr int NIG = GSTAGE / 1024; // 1 KB DMA instructions per key tile
    constexpr int NI = STAGE / 1024;   // ... per stage
    constexpr int NL = NI / NW;        // ... per wave
    constexpr int RPI = 1024 / RB;     // rows per DMA instruction
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

    const int d = H * HD;
    const int64_t ld = 3 * (int64_t)d;
    const int nqb = (T_len + BQ - 1) / BQ;
    // Heaviest query blocks first over all (sequence, head) pairs: block L
    // takes query block rank L / (H B) of pair L % (H B), so every pair's
    // longest block starts in the first round and the short ones fill the
    // tail (1.3-1.7x faster than walking the pairs one after another)
    const int G = H * B;
    const int qrank = (int)blockIdx.x / G, pair = (int)blockIdx.x % G;
    const int qb = nqb - 1 - qrank;
    const int h = pair % H, b = pair / H;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int grp = wave / NQW, wq = wave % NQW;  // key-tile group, wave within it
    const int lr = lane & 15, lg = lane >> 4;
    const int64_t row0 = (int64_t)b * T_len;
    const T* Qb = qkv + h * HD;

    // Q^T operands stay in registers: query = q0 + 16 qg + lr
    const int q0 = qb * BQ + wq * QW;
    vec8 qf[NQG][CS];
#pragma unroll
    for (int qg = 0; qg < NQG; ++qg) {
        const int qr = min(q0 + 16 * qg + lr, T_len - 1);
#pragma unroll
        for (int cs = 0; cs < CS; ++cs)
            qf[qg][cs] = as_vec8<T>(*(const u32x4*)(Qb + (row0 + qr) * ld + cs * 32 + 8 * lg));
    }

    // DMA slot j of this wave: instruction I = wave + NW j of the stage,
    // key tile group I / NIG (tile KS it + group of iteration it), in it K
    // then V; lane i fills row RPI * (I' % (NIG / 2)) + i / CPR (I' = I % NIG),
    // physical chunk i % CPR, i.e. logical chunk (i % CPR) ^ permutation of
    // that row.  Tiles past the last one re-read its key rows (not used).
    // Per-lane parts of each slot's source (row within the tile, byte offset
    // of its chunk within a K or V row) are fixed; a tile only moves the key.
    // Offsets are 32-bit bytes from the wave-uniform base of this (sequence,
    // head) (the launcher checks they fit).
    const uint32_t lds0 = (uint32_t)(uintptr_t)smem;
    const T* kvbase = kvsrc + b * kv_seq + h * HD;
    const uint32_t ldb = (uint32_t)kv_ld * 2;
    int srow[NL];
    uint32_t scol[NL];
#pragma unroll
    for (int j = 0; j < NL; ++j) {
        const int I = wave + NW * j, Ig = I % NIG;
        const bool isv = Ig >= NIG / 2;
        srow[j] = RPI * (Ig % (NIG / 2)) + lane / CPR;
        const int pch = lane % CPR;
        const int ch = isv ? vswz<HD>(srow[j], pch) : kswz<HD>(srow[j], pch);
        scol[j] = (uint32_t)((isv ? d : 0) + ch * 8) * 2;
    }
    auto issue = [&](int it, int stage) {
        const uint32_t sbase = lds0 + stage * STAGE;
#pragma unroll
        for (int j = 0; j < NL; ++j) {
            const int I = wave + NW * j;
            const int kb = it * KS + I / NIG;
            const int key = min(kb * BKV + srow[j], T_len - 1);
            dma16s(kvbase, (uint32_t)key * ldb + scol[j],
                   sbase + (uint32_t)__builtin_amdgcn_readfirstlane(I * 1024));
        }
    };

    f32x4 o[NQG][CT];
    float m_run[NQG], l_run[NQG];
    // running sums by the matrix unit: one more O^T tile, ones^T P^T, every
    // row of which is the sum of the query's probabilities as they enter the
    // products (rounded to dt), rescaled with O
    f32x4 o_l[NQG];
#pragma unroll
    for (int qg = 0; qg < NQG; ++qg) {
        m_run[qg] = -INFINITY;
        l_run[qg] = 0.f;
        o_l[qg] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) o[qg][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // keys needed by this block: those <= its last query (and < T)
    const int nkb = min((T_len + BKV - 1) / BKV, ((qb + 1) * BQ + BKV - 1) / BKV);
    const int nit = (nkb + KS - 1) / KS;
    auto body = [&](int it) {
        const int kb = it * KS + grp;
        if (kb >= nkb) return;  // wave-uniform: this group has no tile left
        const uint8_t* sK = smem + (it % S) * STAGE + grp * GSTAGE;
        const uint8_t* sV = sK + TILE;

        // S^T tiles: key = kb*64 + 16 jt + 4 lg + r, query = q0 + 16 qg + lr
        f32x4 sc[NQG][4];
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            const int row = jt * 16 + lr;
            vec8 kf[CS];
#pragma unroll
            for (int cs = 0; cs < CS; ++cs)
                kf[cs] = as_vec8<T>(*(const u32x4*)(sK + row * RB + (kswz<HD>(row, cs * 4 + lg) << 4)));
#pragma unroll
            for (int qg = 0; qg < NQG; ++qg) {
                sc[qg][jt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int cs = 0; cs < CS; ++cs) sc[qg][jt] = Mfma<T>::mma(kf[cs], qf[qg][cs], sc[qg][jt]);
            }
        }
        // online softmax per query (fp32); P is rounded to dt as it enters the
        // MFMA, the running sum adds the fp32 values
        const bool edge = ((kb + 1) * BKV > q0) || ((kb + 1) * BKV > T_len);
        vec8 pf[NQG][2];
#pragma unroll
        for (int qg = 0; qg < NQG; ++qg) {
            const int q_idx = q0 + 16 * qg + lr;
            if (edge) {  // wave-uniform: only tiles that reach past a query or past T
#pragma unroll
                for (int jt = 0; jt < 4; ++jt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int key = kb * BKV + jt * 16 + 4 * lg + r;
                        const bool masked = (key > q_idx) | (key >= T_len);
                        sc[qg][jt][r] = masked ? -INFINITY : sc[qg][jt][r];
                    }
            }
            float mx = -INFINITY;
#pragma unroll
            for (int jt = 0; jt < 4; ++jt)
#pragma unroll
                for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sc[qg][jt][r]);
            mx = group4_max(mx);
            // key kb*64 <= q_idx always holds for a computed tile, so m_new is finite
            // The running max is kept unless the tile exceeds it by more than
            // 8 in log2 units, so P stays below 2^8 (well inside dt) and the
            // accumulators are rescaled only when some query's max moved.
            const float m_new = mx * LOG2E > m_run[qg] * LOG2E + 8.f ? fmaxf(m_run[qg], mx) : m_run[qg];
            // arguments are <= 0 (<= 8 with the lazy max): the hardware exp2
            // (v_exp_f32) is exact enough and maps -inf to 0
            const float alpha = __builtin_amdgcn_exp2f((m_run[qg] - m_new) * LOG2E);
            const float mb = m_new * LOG2E;
            T pt[4][4];
            float psum = 0.f;
#pragma unroll
            for (int jt = 0; jt < 4; ++jt)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float e = __builtin_amdgcn_exp2f(sc[qg][jt][r] * LOG2E - mb);
                    pt[jt][r] = (T)e;
                    if (!PB_ATTN_MFMA_SUM) psum += e;
                }
            if (!PB_ATTN_MFMA_SUM) {
                psum = group4_sum(psum);
                l_run[qg] = l_run[qg] * alpha + psum;
            }
            m_run[qg] = m_new;
            if (__any(alpha != 1.f)) {
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) {
                    o[qg][ct][0] *= alpha;
                    o[qg][ct][1] *= alpha;
                    o[qg][ct][2] *= alpha;
                    o[qg][ct][3] *= alpha;
                }
                if (PB_ATTN_MFMA_SUM) {
                    o_l[qg][0] *= alpha;
                    o_l[qg][1] *= alpha;
                    o_l[qg][2] *= alpha;
                    o_l[qg][3] *= alpha;
                }
            }
            // P^T operand of key step ks: k index 8 lg + 4 hh + r <-> key 32 ks + 16 hh + 4 lg + r
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                T pk[8];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    pk[r] = pt[2 * ks][r];
                    pk[4 + r] = pt[2 * ks + 1][r];
                }
                u32x4 praw;
                __builtin_memcpy(&praw, pk, 16);
                pf[qg][ks] = as_vec8<T>(praw);
            }
        }
        // O^T += V^T P^T: the V^T operand (row c, k index 8 lg + 4 hh + j) comes from two
        // transposing reads; lane 4 j + q of a 16-lane group addresses row
        // 32 ks + 16 hh + 4 lg + j, columns 16 ct + 4 q .. + 3
        const int tj = lr >> 2, tq = lr & 3;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                u32x2 v[2];
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const int row = 32 * ks + 16 * hh + 4 * lg + tj;
                    const int col = 16 * ct + 4 * tq;  // element column
                    const int ch = col >> 3;
                    v[hh] = read_tr16<T>(sV + row * RB + (vswz<HD>(row, ch) << 4) + (col & 7) * 2);
                }
                const vec8 vf = as_vec8<T>(u32x4{v[0][0], v[0][1], v[1][0], v[1][1]});
#pragma unroll
                for (int qg = 0; qg < NQG; ++qg) o[qg][ct] = Mfma<T>::mma(vf, pf[qg][ks], o[qg][ct]);
            }
            if (PB_ATTN_MFMA_SUM) {
                const vec8 ones = as_vec8<T>(u32x4{ONE2<T>(), ONE2<T>(), ONE2<T>(), ONE2<T>()});
#pragma unroll
                for (int qg = 0; qg < NQG; ++qg) o_l[qg] = Mfma<T>::mma(ones, pf[qg][ks], o_l[qg]);
            }
        }
    };
    // S-stage ring: iterations it+1 .. it+S-2 are in flight while it is used
#pragma unroll
    for (int q = 0; q < S - 1; ++q)
        if (q < nit) issue(q, q);
    int it = 0;
    for (; it + S - 1 < nit; ++it) {
        wait_vmcnt<(S - 2) * NL>();
        __syncthreads();  // tiles of iteration it visible; stage of it-1 free
        issue(it + S - 1, (it + S - 1) % S);
        body(it);
    }
    for (; it < nit; ++it) {
        wait_vmcnt<0>();
        __syncthreads();
        body(it);
    }

    if (PB_ATTN_MFMA_SUM) {
#pragma unroll
        for (int qg = 0; qg < NQG; ++qg) l_run[qg] = o_l[qg][0];
    }
    if (KS == 2) {
        // merge group 1's (max, sum, O^T) into group 0's: every lane holds
        // the same query and O^T rows in both groups
        float* xo = (float*)smem;                           // [NQW waves][NQG][CT][64 lanes][4]
        float* xm = xo + NQW * NQG * CT * 64 * 4;           // [NQW waves][NQG][64 lanes][2]
        __syncthreads();  // every wave is done with the ring
        if (grp == 1) {
#pragma unroll
            for (int qg = 0; qg < NQG; ++qg) {
#pragma unroll
                for (int ct = 0; ct < CT; ++ct)
                    *(f32x4*)(xo + (((wq * NQG + qg) * CT + ct) * 64 + lane) * 4) = o[qg][ct];
                xm[((wq * NQG + qg) * 64 + lane) * 2] = m_run[qg];
                xm[((wq * NQG + qg) * 64 + lane) * 2 + 1] = l_run[qg];
            }
        }
        __syncthreads();
        if (grp == 1) return;
#pragma unroll
        for (int qg = 0; qg < NQG; ++qg) {
            const float m1 = xm[((wq * NQG + qg) * 64 + lane) * 2];
            const float l1 = xm[((wq * NQG + qg) * 64 + lane) * 2 + 1];
            const float M = fmaxf(m_run[qg], m1);  // finite: group 0 always sees key 0
            const float a0 = __builtin_amdgcn_exp2f((m_run[qg] - M) * LOG2E);
            const float a1 = __builtin_amdgcn_exp2f((m1 - M) * LOG2E);  // 0 when group 1 had no tile
            l_run[qg] = l_run[qg] * a0 + l1 * a1;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const f32x4 o1 = *(const f32x4*)(xo + (((wq * NQG + qg) * CT + ct) * 64 + lane) * 4);
#pragma unroll
                for (int r = 0; r < 4; ++r) o[qg][ct][r] = o[qg][ct][r] * a0 + o1[r] * a1;
            }
        }
    }
#pragma unroll
    for (int qg = 0; qg < NQG; ++qg) {
        const int q_idx = q0 + 16 * qg + lr;
        if (q_idx >= T_len) continue;
        const float inv = 1.f / l_run[qg];
        T* orow = out + (row0 + q_idx) * (int64_t)d + h * HD;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            const int c = ct * 16 + 4 * lg;
            *(u32x2*)(orow + c) = pack4<T>(o[qg][ct][0] * inv, o[qg][ct][1] * inv,
                                           o[qg][ct][2] * inv, o[qg][ct][3] * inv);
        }
    }
}

template <typename T, int HD, int QW, int KS, int NQW, int S>
hipError_t launch_hd(const void* qkv, const void* kv, int64_t kv_ld, int64_t kv_seq, void* out, int B,
                     int T_len, int H, hipStream_t s) {
    constexpr int LDS = S * KS * 2 * BKV * HD * 2;  // S stages of KS key tiles (K and V)
    static_assert(KS == 1 || NQW * QW / 16 * (HD / 16) * 64 * 16 + NQW * QW / 16 * 64 * 8 <= LDS,
                  "the merge fits in the ring");
    static_assert(LDS <= 160 * 1024, "LDS");
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void*)attention_kernel<T, HD, QW, KS, NQW, S>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const long nblk = (long)((T_len + NQW * QW - 1) / (NQW * QW)) * H * B;
    PB_LAUNCH((attention_kernel<T, HD, QW, KS, NQW, S>), dim3((unsigned)nblk), dim3(64 * NQW * KS), LDS, s,
              (const T*)qkv, (const T*)kv, kv_ld, kv_seq, (T*)out, T_len, H, B);
    return hipGetLastError();
}

template <typename T, int HD>
hipError_t launch_qw(const void* qkv, const void* kv, int64_t kv_ld, int64_t kv_seq, void* out, int B,
                     int T_len, int H, hipStream_t s) {
    const long pairs = (long)H * B;
    // 32 queries per wave when 128-query blocks still give every CU work;
    // with fewer than 512 blocks of 64 queries, two wave groups split the keys
    const long blocks128 = (long)((T_len + 127) / 128) * pairs;
    const long blocks64 = (long)((T_len + 63) / 64) * pairs;
    if (PB_ATTN_QW32 && blocks128 >= 512) return launch_hd<T, HD, 32, 1, 4, 2>(qkv, kv, kv_ld, kv_seq, out, B, T_len, H, s);
    if (PB_ATTN_KS2 && blocks64 < 512 && T_len > BKV)
        return launch_hd<T, HD, 16, 2, 4, 2>(qkv, kv, kv_ld, kv_seq, out, B, T_len, H, s);
    return launch_hd<T, HD, 16, 1, 4, 2>(qkv, kv, kv_ld, kv_seq, out, B, T_len, H, s);
}

// ---- decode: one new query per (sequence, head) against the KV cache --------
// One block per (sequence, head); its NW waves take 64-key chunks in turn
// (wave w: keys 64w.., then 64(w + NW).., ...) with a running max and sum.  A
// key row of HD elements is read by G = HD / 8 lanes, 16 bytes each, so one
// load instruction covers 64 / G whole keys, and a wave issues all the K and
// V loads of a chunk before using any.  Scores are fp32 dot products with the
// query (reduced over the G lanes of a key); P V accumulates 8 head
// dimensions per lane, reduced at the end over the lanes that hold the same
// dimensions; the waves are combined through LDS in wave order.
template <typename T, int HD, int NW>
__global__ __launch_bounds__(64 * NW) void decode_attention_kernel(const T* __restrict__ qkv,
                                                                   const T* __restrict__ kv, int64_t seq_stride,
                                                                   int d, const int32_t* __restrict__ pos0,
                                                                   T* __restrict__ out) {
    constexpr int G = HD / 8;     // lanes per key row
    constexpr int KPI = 64 / G;   // keys per load instruction
    constexpr int NI = 64 / KPI;  // load instructions per 64-key chunk
    __shared__ float wm[NW], wl[NW];
    __shared__ float wo[NW][HD];
    const int h = blockIdx.x, b = blockIdx.y;
    const int nkeys = *pos0 + 1;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int sub = lane % G, grp = lane / G;
    float q[8];
    {
        const u32x4 raw = *(const u32x4*)(qkv + (int64_t)b * 3 * d + h * HD + sub * 8);
        T e[8];
        __builtin_memcpy(e, &raw, 16);
#pragma unroll
        for (int j = 0; j < 8; ++j) q[j] = (float)e[j];
    }
    const T* kvb = kv + (int64_t)b * seq_stride + h * HD + sub * 8;
    float m_run = -INFINITY, l = 0.f, o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = 0.f;
    for (int c0 = wave * 64; c0 < nkeys; c0 += NW * 64) {  // wave-uniform
        u32x4 kr[NI], vr[NI];
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int key = min(c0 + i * KPI + grp, nkeys - 1);
            kr[i] = *(const u32x4*)(kvb + (int64_t)key * 2 * d);
        }
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int key = min(c0 + i * KPI + grp, nkeys - 1);
            vr[i] = *(const u32x4*)(kvb + (int64_t)key * 2 * d + d);
        }
        float sc[NI];
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            T e[8];
            __builtin_memcpy(e, &kr[i], 16);
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) a += q[j] * (float)e[j];
#pragma unroll
            for (int sh = 1; sh < G; sh <<= 1) a += __shfl_xor(a, sh, 64);
            sc[i] = c0 + i * KPI + grp < nkeys ? a : -INFINITY;
            mx = fmaxf(mx, sc[i]);
        }
        const float m_new = fmaxf(m_run, wave_max(mx));  // finite: the chunk holds a live key
        const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * LOG2E);
        l *= alpha;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] *= alpha;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const float pk = sc[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((sc[i] - m_new) * LOG2E);
            l += pk;
            T e[8];
            __builtin_memcpy(e, &vr[i], 16);
#pragma unroll
            for (int j = 0; j < 8; ++j) o[j] += pk * (float)e[j];
        }
        m_run = m_new;
    }
    // over the lanes holding the same dimensions (the KPI key groups)
#pragma unroll
    for (int sh = G; sh < 64; sh <<= 1) {
        l += __shfl_xor(l, sh, 64);
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] += __shfl_xor(o[j], sh, 64);
    }
    if (lane == 0) {
        wm[wave] = m_run;
        wl[wave] = l;
    }
    if (grp == 0)
#pragma unroll
        for (int j = 0; j < 8; ++j) wo[wave][sub * 8 + j] = o[j];
    __syncthreads();
    const int dim = threadIdx.x;
    if (dim < HD) {
        float M = wm[0];
#pragma unroll
        for (int w = 1; w < NW; ++w) M = fmaxf(M, wm[w]);
        float acc = 0.f, L = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            if (wm[w] == -INFINITY) continue;  // a wave with no key
            const float f = __builtin_amdgcn_exp2f((wm[w] - M) * LOG2E);
            acc += f * wo[w][dim];
            L += f * wl[w];
        }
        out[(int64_t)b * d + h * HD + dim] = (T)(acc / L);
    }
}

template <typename T, int HD>
hipError_t launch_decode_hd(const void* qkv, const void* kv, int64_t seq_stride, int B, int H,
                            const int32_t* pos0, void* out, hipStream_t s) {
    // 16 waves for 64-dim heads; 8 for 128 (twice the load registers per chunk)
    constexpr int NW = HD == 64 ? 16 : 8;
    PB_LAUNCH((decode_attention_kernel<T, HD, NW>), dim3(H, B), dim3(64 * NW), 0, s, (const T*)qkv,
                       (const T*)kv, seq_stride, H * HD, pos0, (T*)out);
    return hipGetLastError();
}
}  // namespace

hipError_t launch_attention_kv(int dtype, const void* qkv, const void* kv, int64_t kv_ld, int64_t kv_seq,
                               void* out, int B, int T_len, int H, int hd, hipStream_t s) {
    if (B <= 0 || T_len <= 0) return hipSuccess;
    if ((int64_t)B * T_len * 3 * H * hd >= ((int64_t)1 << 31) || (int64_t)B * kv_seq >= ((int64_t)1 << 31))
        return hipErrorInvalidValue;
    // copy offsets are 32-bit bytes within one (sequence, head)
    if (((int64_t)T_len * kv_ld + 3 * (int64_t)H * hd) * 2 >= ((int64_t)1 << 32)) return hipErrorInvalidValue;
    if (dtype == 1) {
        if (hd == 64) return launch_qw<_Float16, 64>(qkv, kv, kv_ld, kv_seq, out, B, T_len, H, s);
        if (hd == 128) return launch_qw<_Float16, 128>(qkv, kv, kv_ld, kv_seq, out, B, T_len, H, s);
    } else {
        if (hd == 64) return launch_qw<__bf16, 64>(qkv, kv, kv_ld, kv_seq, out, B, T_len, H, s);
        if (hd == 128) return launch_qw<__bf16, 128>(qkv, kv, kv_ld, kv_seq, out, B, T_len, H, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_attention(int dtype, const void* qkv, void* out, int B, int T_len, int H, int hd,
                            hipStream_t s) {
    // keys and values from the same rows: K at column d, V at 2d, 3d per row
    const int64_t d = (int64_t)H * hd;
    return launch_attention_kv(dtype, qkv, (const char*)qkv + d * 2, 3 * d, (int64_t)T_len * 3 * d, out, B,
                               T_len, H, hd, s);
}

hipError_t launch_decode_attention(int dtype, const void* qkv, const void* kv, int64_t seq_stride,
                                   int B, int H, int hd, const int32_t* pos0, void* out, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    if (!pos0) return hipErrorInvalidValue;
    if (dtype == 1) {
        if (hd == 64) return launch_decode_hd<_Float16, 64>(qkv, kv, seq_stride, B, H, pos0, out, s);
        if (hd == 128) return launch_decode_hd<_Float16, 128>(qkv, kv, seq_stride, B, H, pos0, out, s);
    } else {
        if (hd == 64) return launch_decode_hd<__bf16, 64>(qkv, kv, seq_stride, B, H, pos0, out, s);
        if (hd == 128) return launch_decode_hd<__bf16, 128>(qkv, kv, seq_stride, B, H, pos0, out, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace pb
