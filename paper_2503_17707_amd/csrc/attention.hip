// Causal self-attention of the prefill (Section 2.1: every layer relates all
// prompt tokens through self-attention; a prefill is causal, token j sees
// tokens 0..j), flash-style: the T x T score matrix is never stored.
//
// Block = 4 waves = 64 queries of one (sequence, head); each wave owns 16
// queries.  Key/value blocks of 64 rows are staged in LDS (K row-major, V
// transposed) and consumed with v_mfma_f32_16x16x32_{f16,bf16}:
//
//   S^T[key, query] = K Q^T      A operand = K rows, B operand = the wave's Q
//                                 (held in registers for the whole kernel)
//   O^T[c, query]  += V^T P^T    A operand = V^T rows, B operand = P^T
//
// With the transposed products every lane holds scores and outputs of one
// query (lane % 16), so the online softmax (running max m, running sum l, in
// fp32) needs only cross-lane reductions over the 4 lane groups and no
// transposition of P: the 8 keys a lane contributes to one P^T operand are the
// 8 scores it already holds, and V^T is read in the same key order.
//
// Blocks run heaviest-first (the last query block sees the most keys).
#include "common.h"
#include "kernels.h"

namespace pb {

namespace {

constexpr float LOG2E = 1.4426950408889634f;

template <int HD>
__device__ __forceinline__ int kswz(int row, int ch) {
    // K tile rows are HD*2 bytes = HD/8 chunks of 16 bytes
    if (HD == 64) return ch ^ (row & 7);
    return ch ^ (row & 15);
}

template <typename T, int HD>
__global__ __launch_bounds__(256) void attention_kernel(const T* __restrict__ qkv,
                                                       T* __restrict__ out, int T_len, int H) {
    typedef typename Mfma<T>::vec8 vec8;
    constexpr int BQ = 64, BKV = 64;
    constexpr int CS = HD / 32;   // 32-wide k steps over head_dim
    constexpr int CT = HD / 16;   // 16-row tiles of O^T
    constexpr int KCH = HD / 8;   // 16-byte chunks per K row
    __shared__ __attribute__((aligned(16))) uint8_t sK[BKV * HD * 2];
    __shared__ __attribute__((aligned(16))) uint8_t sV[HD * BKV * 2];  // V^T: [HD][64 keys]

    const int d = H * HD;
    const int64_t ld = 3 * (int64_t)d;
    const int nqb = (T_len + BQ - 1) / BQ;
    const int qb = nqb - 1 - (int)blockIdx.x;
    const int h = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    const int64_t row0 = (int64_t)b * T_len;
    const T* Qb = qkv + h * HD;
    const T* Kb = qkv + d + h * HD;
    const T* Vb = qkv + 2 * d + h * HD;

    const int q_idx = qb * BQ + wave * 16 + lr;
    const int q_row = min(q_idx, T_len - 1);
    vec8 qf[CS];
#pragma unroll
    for (int cs = 0; cs < CS; ++cs)
        qf[cs] = as_vec8<T>(*(const u32x4*)(Qb + (row0 + q_row) * ld + cs * 32 + 8 * lg));

    f32x4 o[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) o[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    const int nkb = qb + 1;
    for (int kb = 0; kb < nkb; ++kb) {
        __syncthreads();
        // stage K (row-major, swizzled) and V^T (swizzled 8-byte units)
#pragma unroll
        for (int i = 0; i < BKV * KCH / 256; ++i) {
            const int c = tid + 256 * i, row = c / KCH, ch = c % KCH;
            const int key = min(kb * BKV + row, T_len - 1);
            const u32x4 kv = *(const u32x4*)(Kb + (row0 + key) * ld + ch * 8);
            *(u32x4*)(sK + row * HD * 2 + (kswz<HD>(row, ch) << 4)) = kv;
            const u32x4 vv = *(const u32x4*)(Vb + (row0 + key) * ld + ch * 8);
            T ve[8];
            __builtin_memcpy(ve, &vv, 16);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int cc = ch * 8 + e;  // column of V = row of V^T
                const int unit = (row >> 2) ^ (cc & 15);
                *(T*)(sV + cc * (BKV * 2) + unit * 8 + (row & 3) * 2) = ve[e];
            }
        }
        __syncthreads();

        // S^T tiles: key = kb*64 + 16*jt + 4*lg + r, query = q_idx
        f32x4 s[4];
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            s[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
            const int row = jt * 16 + lr;
#pragma unroll
            for (int cs = 0; cs < CS; ++cs) {
                const int ch = cs * 4 + lg;
                const vec8 kf = as_vec8<T>(*(const u32x4*)(sK + row * HD * 2 + (kswz<HD>(row, ch) << 4)));
                s[jt] = Mfma<T>::mma(kf, qf[cs], s[jt]);
            }
        }
        // mask (causal and ragged tail) and block maximum
        float mx = -INFINITY;
        const bool diag = (kb == qb) || ((kb + 1) * BKV > T_len);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int key = kb * BKV + jt * 16 + 4 * lg + r;
                if (diag && (key > q_idx || key >= T_len)) s[jt][r] = -INFINITY;
                mx = fmaxf(mx, s[jt][r]);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run, mx);  // finite: key kb*64 <= q_idx is always allowed
        const float alpha = exp2f((m_run - m_new) * LOG2E);
        const float mb = m_new * LOG2E;
        // probabilities, rounded to dt as they enter the MFMA; the sum uses the rounded values
        T pt[4][4];
        float psum = 0.f;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const T pv = (T)exp2f(s[jt][r] * LOG2E - mb);
                pt[jt][r] = pv;
                psum += (float)pv;
            }
        psum += __shfl_xor(psum, 16, 64);
        psum += __shfl_xor(psum, 32, 64);
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            o[ct][0] *= alpha;
            o[ct][1] *= alpha;
            o[ct][2] *= alpha;
            o[ct][3] *= alpha;
        }
        // O^T += V^T P^T over two 32-key steps; k index 8*lg + 4*hh + r <-> key 32*ks + 16*hh + 4*lg + r
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
            const vec8 pf = as_vec8<T>(praw);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const int cc = ct * 16 + lr;
                const int u0 = ((32 * ks + 4 * lg) >> 2) ^ (cc & 15);
                const int u1 = ((32 * ks + 16 + 4 * lg) >> 2) ^ (cc & 15);
                const u32x2 v0 = *(const u32x2*)(sV + cc * (BKV * 2) + u0 * 8);
                const u32x2 v1 = *(const u32x2*)(sV + cc * (BKV * 2) + u1 * 8);
                const u32x4 vraw = u32x4{v0[0], v0[1], v1[0], v1[1]};
                o[ct] = Mfma<T>::mma(as_vec8<T>(vraw), pf, o[ct]);
            }
        }
    }

    if (q_idx < T_len) {
        const float inv = 1.f / l_run;
        T* orow = out + (row0 + q_idx) * (int64_t)d + h * HD;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            const int c = ct * 16 + 4 * lg;
            *(u32x2*)(orow + c) = pack4<T>(o[ct][0] * inv, o[ct][1] * inv, o[ct][2] * inv,
                                           o[ct][3] * inv);
        }
    }
}

template <typename T, int HD>
hipError_t launch_hd(const void* qkv, void* out, int B, int T_len, int H, hipStream_t s) {
    dim3 grid((T_len + 63) / 64, H, B);
    hipLaunchKernelGGL((attention_kernel<T, HD>), grid, dim3(256), 0, s, (const T*)qkv, (T*)out,
                       T_len, H);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(int dtype, const void* qkv, void* out, int B, int T_len, int H,
                            int hd, hipStream_t s) {
    if (B <= 0 || T_len <= 0) return hipSuccess;
    if (dtype == 1) {
        if (hd == 64) return launch_hd<_Float16, 64>(qkv, out, B, T_len, H, s);
        if (hd == 128) return launch_hd<_Float16, 128>(qkv, out, B, T_len, H, s);
    } else {
        if (hd == 64) return launch_hd<__bf16, 64>(qkv, out, B, T_len, H, s);
        if (hd == 128) return launch_hd<__bf16, 128>(qkv, out, B, T_len, H, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace pb
