// Launch wrappers of the CDNA4 kernels (host-callable, plain pointers).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rowops.h"

namespace pb {

enum GemmEpilogue {
    EPI_QKV = 0,     // C = dt((acc + bias) * (n < qcols ? qscale : 1))
    EPI_RELU = 1,    // C = dt(max(acc + bias, 0))
    EPI_RESID = 2,   // R += acc + bias            (fp32 residual stream)
    EPI_SHRINK = 3,  // C = dt(acc * slot_scale[s]) if column block (n % kw) / slot_width == s,
                     //     s = row_slot[m] >= 0; 0 otherwise
};

// Y[M, N] = X[M, K1] W[N, K1]^T (+ X2[M, K2] W2[N, K2]^T) followed by an epilogue.
// X, W, X2, W2 are row-major with the reduction dimension contiguous.  The
// optional second segment is the LoRA expand: for an N tile starting at n0 it
// is active when bit (n0 / group) of k2_mask is set, and then reads X2 at
// column offset (n0 / group) * x2_group_stride.  K1 and K2 are multiples of
// 64, N a multiple of 64; M is arbitrary (ragged tails are masked).
struct GemmParams {
    const void* X; int64_t ldx;
    const void* W; int64_t ldw;
    int M, N, K1;
    const void* X2; int64_t ldx2;
    const void* W2; int64_t ldw2;
    int K2; int group; uint32_t k2_mask; int64_t x2_group_stride;
    const void* bias;
    void* C; int64_t ldc;
    float* R; int64_t ldr;
    float qscale; int qcols;
    // Optional KV-cache write (EPI_QKV): the key and value columns [qcols,
    // 3 qcols) of token row m also go to cache row (m / kv_T) * kv_seq +
    // (*kv_pos + m % kv_T) * 2 qcols, laid out [k | v] (kv NULL = none).
    void* kv; const int32_t* kv_pos; int kv_T; int64_t kv_seq;
    const int32_t* row_slot; const float* slot_scale; int slot_width; int kw;
    // Optional LayerNorm fused after a residual epilogue (EPI_RESID with N the
    // model width): when the launcher splits K, its row-wise reduce also writes
    // ln_out = dt(LN(R) * ln_g + ln_b) and sets *ln_done.
    const void* ln_g; const void* ln_b; void* ln_out; float ln_eps; bool* ln_done;
    // Optional LoRA shrink of the fused LayerNorm's rows (Acat NULL = none).
    RowShrink shrink;
};

// Device scratch for split-K partials (fp32 [splits][M][N]); splitting is
// skipped when it is absent or too small.
struct GemmWorkspace {
    void* ws;
    size_t bytes;
};

// Products with at most this many token rows stream the weights with the
// GEMV kernel (decode steps) instead of MFMA tiles.
constexpr int GEMV_MAX_ROWS = 8;

// role: 0 qkv, 1 o, 2 fc1, 3 fc2, 4 shrink (selects the instantiation; each
// role has its own kernel symbol so profiles separate them).  Requires every
// operand offset (rows * leading dimension) to fit in 31 bits.
hipError_t launch_gemm(int dtype, int role, int epi, const GemmParams& p, const GemmWorkspace& ws,
                       hipStream_t s);

// Causal multi-head self-attention over a batch of equal-length sequences.
// qkv: [B*T, 3d] (q already divided by sqrt(head_dim)); out: [B*T, d].
hipError_t launch_attention(int dtype, const void* qkv, void* out, int B, int T, int H, int hd,
                            hipStream_t s);
// The same with keys and values elsewhere: key of (sequence b, position t) at
// kv + b * kv_seq + t * kv_ld (+ h * hd), its value d elements further.
hipError_t launch_attention_kv(int dtype, const void* qkv, const void* kv, int64_t kv_ld, int64_t kv_seq,
                               void* out, int B, int T, int H, int hd, hipStream_t s);

// x[b*T + t, :] = E[tok[b*T + t], :] + P[pos0 + t, :] (fp32 output), with
// pos0 read from device memory (*pos0) so that replays of a recorded launch
// can move it.
hipError_t launch_embed(int dtype, const int32_t* tok, const void* E, const void* P, float* x,
                        int n_rows, int T, int d, const int32_t* pos0, hipStream_t s);

// One new query per (sequence, head) of qkv ([B, 3d], q pre-scaled) against
// cache positions 0 .. *pos0 of kv ([B][seq_stride], rows [k | v] of 2d), the
// last one the new token's own; out [B, d].  The launch does not depend on
// *pos0, so one recorded launch serves every step.
hipError_t launch_decode_attention(int dtype, const void* qkv, const void* kv, int64_t seq_stride,
                                   int B, int H, int hd, const int32_t* pos0, void* out, hipStream_t s);

// out[r, :] = LN(x[r * in_mul + in_add, :]) * g + b, fp32 statistics;
// out_f32 selects a float output, otherwise dt.
// With sh (dt output only), also writes the row-wise LoRA shrink of each row.
hipError_t launch_layernorm(int dtype, const float* x, int64_t in_mul, int64_t in_add,
                            const void* g, const void* b, void* out, bool out_f32, int rows,
                            int d, float eps, hipStream_t s, const RowShrink* sh = nullptr);

// logits[b, v] = z[b, :] . E[v, :] (fp32 accumulate), plus per-block argmax
// partials pval/pidx [B][lm_head_blocks(V)] (maximum, lowest index on ties);
// d a multiple of 8, at most 16384.
int lm_head_blocks(int V);
hipError_t launch_lm_head(int dtype, const float* z, int B, const void* E, int V, int d,
                          float* logits, float* pval, int* pidx, hipStream_t s);

// tok[b] = lowest index of the maximum of logits[b, :], from the LM head's
// partials (-1 if no finite maximum exists).
hipError_t launch_argmax(const float* pval, const int* pidx, int B, int V, int32_t* tok,
                         hipStream_t s);

// Scatter one adapter's staged LoRA blobs (per layer: A_t [r, d], B_t [d, r] for
// the targets in mask) into slot `slot` of the packed per-layer arrays
// Acat [L][4][kw][d] and Bcat [L][4][d][kw] (slot columns slot*rs .. +rs),
// zero-filling ranks r..rs-1 and absent targets.
// W [d, d] += scale * (slot's B [d, rs]) (slot's A [rs, d]), rounded once (misc.hip).
hipError_t launch_lora_merge(int dtype, void* W, const void* Acat, const void* Bcat, int d, int kw, int rs,
                             int slot, float scale, hipStream_t s);

hipError_t launch_lora_pack(int dtype, const void* staging, size_t staging_layer_elems, int L,
                            int d, int r, uint32_t mask, int slot, int rs, int kw, void* Acat,
                            void* Bcat, hipStream_t s);

}  // namespace pb
