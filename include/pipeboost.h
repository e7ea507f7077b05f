/*
 * pipeboost.h -- C ABI of the MI355X cold-start prefill library.
 *
 * The library runs the prefill of an OPT-style pre-LayerNorm decoder with
 * unmerged LoRA adapters on a shared base model and returns the greedy first
 * token (PipeBoost, arXiv 2503.17707, Section 2.1: prefill through every
 * layer, the last layer yields the first token; LoRA keeps W fixed and adds a
 * low-rank pair A, B).  Its point is the paper's overlap of model loading with
 * inference (Sections 1, 4.2 and 4.3): layer weights stream host-to-device on
 * a copy stream and each layer's compute starts as soon as that layer has
 * landed, gated on the device by one event per layer, while later layers are
 * still in flight.
 *
 * Conventions
 *  - Every function returns a pb_status (0 = PB_OK) unless it returns a size.
 *    Nothing throws across the ABI.  On failure pb_last_error() returns a
 *    thread-local message describing the last failure of the calling thread.
 *  - "dt" below is the model's storage type: bfloat16 (PB_BF16) or IEEE
 *    binary16 (PB_F16).  Every matrix is stored row-major [out, in] (the
 *    reduction dimension contiguous).  Tensor offsets are in elements of dt.
 *  - Streams are hipStream_t handles passed as void*.  The caller owns them,
 *    and the device arena; the library sub-allocates the arena and never
 *    frees it.  The library owns its events and a small pinned staging area.
 *  - A model is not thread-safe: use one model per host thread.
 *  - Supported shapes: d_model a multiple of 128 (<= 16384), d_ffn a multiple
 *    of 64, head_dim = d_model / n_heads in {64, 128}, max_rank <= 64,
 *    max_adapters <= 16.
 */
#ifndef PIPEBOOST_H
#define PIPEBOOST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PB_OK = 0,
    PB_EINVAL = -1,      /* bad argument or unsupported shape */
    PB_ENOTPINNED = -2,  /* a host pointer handed to the loader is not pinned */
    PB_ENOMEM = -3,      /* arena too small, or a host allocation failed */
    PB_EHIP = -4,        /* a HIP runtime call failed; pb_last_error() has its message */
    PB_ESTATE = -5       /* call out of order (e.g. prefill before any layer was streamed) */
} pb_status;

typedef enum { PB_BF16 = 0, PB_F16 = 1 } pb_dtype;

/* LoRA target projections (Section 2.1 places adapters on attention weights). */
enum { PB_LORA_Q = 1, PB_LORA_K = 2, PB_LORA_V = 4, PB_LORA_O = 8 };

/* Tensors of one decoder layer blob. */
enum {
    PB_T_LN1_G = 0, PB_T_LN1_B, PB_T_WQ, PB_T_BQ, PB_T_WK, PB_T_BK, PB_T_WV, PB_T_BV,
    PB_T_WO, PB_T_BO, PB_T_LN2_G, PB_T_LN2_B, PB_T_W1, PB_T_B1, PB_T_W2, PB_T_B2,
    PB_T_COUNT
};

/* Tensors of the globals blob: token embedding [vocab, d] (also the tied LM
 * head), learned positions [max_pos, d], final LayerNorm gain and bias [d]. */
enum { PB_G_EMBED = 0, PB_G_POS, PB_G_LNF_G, PB_G_LNF_B, PB_G_COUNT };

typedef struct {
    int32_t n_layers;
    int32_t d_model;
    int32_t n_heads;
    int32_t d_ffn;
    int32_t vocab;
    int32_t max_pos;      /* rows of the position table; a prompt has T <= max_pos */
    int32_t max_tokens;   /* capacity in tokens of one prefill, B * T <= max_tokens */
    int32_t max_batch;    /* capacity in sequences of one prefill */
    int32_t max_adapters; /* LoRA slots */
    int32_t max_rank;     /* largest LoRA rank a slot may hold */
    int32_t dtype;        /* pb_dtype */
    float ln_eps;         /* LayerNorm epsilon (1e-5 for OPT) */
    int32_t max_new_tokens; /* decode steps after a prefill; > 0 keeps a KV cache of
                               [n_layers][max_batch][max_pos][2 d_model] in the arena */
    int32_t merge_shadow;   /* 1: the arena also keeps a copy of every layer's unmerged
                               Wq|Wk|Wv|Wo, so merged adapters can be switched and
                               unmerged on the device (pb_merge_lora, pb_unmerge_lora) */
} pb_config;

typedef struct pb_model pb_model;

/* ---- layout queries (host only; no GPU needed) ------------------------- */

/* Bytes of one layer blob.  The layout is the device execution layout: the
 * loader copies it byte for byte and nothing is converted after landing.
 * Returns 0 if the config is invalid. */
size_t pb_layer_bytes(const pb_config* cfg);

/* Bytes of the globals blob (embedding, positions, final LayerNorm). */
size_t pb_globals_bytes(const pb_config* cfg);

/* Offset (in dt elements) and element count of tensor `tensor` (PB_T_*)
 * inside a layer blob.  wq, wk, wv are consecutive ([3d, d] together) and so
 * are bq, bk, bv.  Every other tensor starts on a 256-byte boundary. */
int pb_layer_tensor(const pb_config* cfg, int32_t tensor, size_t* offset, size_t* numel);

/* Offset and element count of tensor `tensor` (PB_G_*) in the globals blob. */
int pb_globals_tensor(const pb_config* cfg, int32_t tensor, size_t* offset, size_t* numel);

/* Bytes of one layer's LoRA blob for an adapter of rank `rank` on the targets
 * in `target_mask`: for each target present, in the order q, k, v, o, the
 * matrix A [rank, d] (the paper's d x r matrix, transposed) and then B
 * [d, rank] (the paper's r x d matrix, transposed).  Returns 0 if invalid. */
size_t pb_lora_layer_bytes(const pb_config* cfg, int32_t rank, uint32_t target_mask);

/* Offset and element count of A (which = 0) or B (which = 1) of target
 * `target` (0..3 = q, k, v, o) inside such a LoRA layer blob. */
int pb_lora_tensor(const pb_config* cfg, int32_t rank, uint32_t target_mask, int32_t target,
                   int32_t which, size_t* offset, size_t* numel);

/* Device bytes the caller must provide to pb_model_create (weights of every
 * layer, the LoRA slots, activations, staging and scratch). */
size_t pb_arena_bytes(const pb_config* cfg);

/* ---- pinned host memory ------------------------------------------------ */

/* Allocate / free pinned host memory (hipHostMalloc).  Layer blobs in pinned
 * memory are copied by DMA straight from their pages; LoRA blobs must be
 * pinned. */
int pb_host_alloc(size_t bytes, void** out);
int pb_host_free(void* ptr);

/* NUMA node of HIP device `device` (from its PCI address in sysfs), -1 when
 * the system reports none.  PB_EHIP if the device does not exist. */
int pb_host_numa_node(int32_t device, int32_t* node);

/* Place later pb_host_alloc allocations (and the loader's pinned staging
 * ring) on NUMA node `node` (hipHostMallocNumaUser under an MPOL_PREFERRED
 * policy of the calling thread for the duration of the call), or let the runtime
 * choose (-1, the default).  Host memory next to the GPU's PCIe root keeps
 * host-to-device copies off the inter-socket link. */
int pb_set_host_numa_node(int32_t node);

/* ---- model lifecycle ----------------------------------------------------- */

/* Create a model on the current HIP device over the caller's device arena
 * (at least pb_arena_bytes(cfg) bytes, 256-byte aligned).  copy_stream carries
 * every host-to-device transfer; compute_stream carries the forward pass.  The
 * two must differ.  The analog of the paper's "Init Meta" stage (Section 5.2):
 * it validates the config, lays out the arena and zeroes the LoRA slots. */
int pb_model_create(const pb_config* cfg, void* dev_arena, size_t arena_bytes, void* copy_stream,
                    void* compute_stream, pb_model** out);

/* Stream the base model host-to-device (Sections 4.2 and 4.3).  Enqueues on
 * the copy stream, in this order: the globals blob, then layer
 * layer_order[0], layer_order[1], ..., each split into chunks of at most the
 * model's chunk size (pb_set_chunk_bytes), and records one event after each
 * layer's last chunk.  host_layers[l] is layer l's blob (indexed by layer id,
 * not by position in the order); host_globals is the globals blob.  They stay
 * valid and unmodified until the next pb_prefill_first_token returns.
 * layer_order lists n_layers distinct layer ids: all of them (a permutation
 * of the model's layers) or, for a pipeline stage (pb_prefill_stage), a
 * subset; a listed layer's blob must not be NULL (PB_EINVAL otherwise), and a
 * prefill that needs an unlisted layer fails with PB_ESTATE.  Blobs in pinned memory are copied by DMA from their
 * own pages.  If any blob is pageable (hosts may cap locked memory below the
 * model's size), the library copies pageable blobs through its own pinned
 * staging ring (4 x 64 MiB, allocated on first use; PB_ENOMEM if it cannot
 * be) with multi-threaded host copies, on a loader thread that enqueues every
 * blob in the same order; pb_prefill_first_token then waits on the host until
 * each layer's copies are enqueued before it enqueues the wait for that
 * layer.  Returns immediately: the copies are asynchronous.  The layer each
 * position lands in does not depend on the order, and neither do the results
 * of a later prefill.  Errors of the loader thread surface from the next
 * pb_prefill_first_token or pb_last_load_stats. */
int pb_stream_layers(pb_model* m, const int32_t* layer_order, int32_t n_layers,
                     const void* const* host_layers, const void* host_globals);

/* Load a LoRA adapter into slot `slot` (Section 4.2.2: adapters share the base
 * model).  host_lora[l] is layer l's LoRA blob laid out as pb_lora_layer_bytes
 * describes for (rank, target_mask); scale = alpha / rank.  Copies and packs on
 * the copy stream and records an event that the next prefill waits for, so
 * call it before pb_stream_layers for the adapter to land ahead of the base
 * layers.  Host blobs must be pinned.  Replaces whatever the slot held. */
int pb_attach_lora(pb_model* m, int32_t slot, int32_t rank, float alpha, uint32_t target_mask,
                   const void* const* host_lora);

/* Prefill B prompts of T tokens each and return the greedy first token of
 * each (Section 2.1).  tokens: host int32 [B*T], sequence-major, each in
 * [0, vocab).  adapter_of_seq: host int32 [B], the LoRA slot of each sequence
 * or -1 for the base model; NULL means all -1.  out_tokens: host int32 [B].
 * out_logits: host float [B*vocab] (the last position's logits) or NULL.
 * Layers run in natural order 0..L-1 and the compute stream waits on the
 * device for each layer's event, so compute overlaps the copies still in
 * flight.  Blocks until the outputs are in host memory.  Requires
 * 1 <= B <= max_batch, 1 <= T <= max_pos, B*T <= max_tokens, attached slots
 * for every adapter used, and a prior pb_stream_layers (PB_ESTATE).  Ties in
 * the argmax go to the lowest token id. */
int pb_prefill_first_token(pb_model* m, const int32_t* tokens, int32_t B, int32_t T,
                           const int32_t* adapter_of_seq, int32_t* out_tokens, float* out_logits);

/* Decode stage (Section 2.1): one more token for each sequence of the last
 * prefill, attending to the KV cache that prefill and earlier steps filled.
 * tokens: host int32 [B], the newest token of each sequence (the previous
 * call's out_tokens to continue greedily); it takes position T + steps so far
 * and its keys and values join the cache.  adapter_of_seq must equal the
 * prefill's.  out_tokens / out_logits as for the prefill.  Requires a model
 * created with max_new_tokens > 0 and a prior successful prefill of the same
 * B (PB_ESTATE / PB_EINVAL otherwise); at most max_new_tokens steps, and the
 * sequences stay within max_pos positions (PB_ESTATE).  Blocks until the
 * outputs are in host memory. */
int pb_decode_step(pb_model* m, const int32_t* tokens, int32_t B, const int32_t* adapter_of_seq,
                   int32_t* out_tokens, float* out_logits);

/* Pipeline loading plan across GPUs (Sections 4.2.1 and 4.4.2), host only:
 * the layer order each GPU of a server streams, after start-up or after some
 * GPUs failed.  alive[g] != 0 for each of the n_gpus GPUs still running.  The
 * alive GPUs, in index order, own consecutive blocks of layers (balance:
 * sizes differ by at most one, the earlier blocks taking the remainder;
 * contiguity: one run of layers each); GPU g's order lists its block first,
 * then the layers after it, cyclically, so a pipeline over the alive GPUs can
 * start once every block has landed while each GPU goes on to load the whole
 * model.  order: int32 [n_gpus * n_layers], row g a permutation of
 * 0..n_layers-1 for an alive GPU and all -1 for a failed one (pass a row to
 * pb_stream_layers, skipping layers the GPU already holds); block_first,
 * block_len: int32 [n_gpus] or NULL (-1 / 0 for failed GPUs).  With every GPU
 * alive and n_gpus dividing n_layers, GPU g's order is the rotation starting
 * at layer g * n_layers / n_gpus.  PB_EINVAL for bad sizes or no alive GPU. */
int pb_plan_loading(int32_t n_layers, int32_t n_gpus, const uint8_t* alive, int32_t* order,
                    int32_t* block_first, int32_t* block_len);

/* One pipeline stage of a prefill (Sections 4.2.1, 4.3.1: a GPU that holds a
 * contiguous block of layers runs them and hands the hidden states on).
 * Runs layers [layer_begin, layer_end) of B sequences of T tokens.  A stage
 * starting at layer 0 embeds `tokens`; a later one reads the previous
 * stage's hidden state from hidden_in (device, fp32 [B*T][d_model], row b*T+t).
 * A stage ending before the last layer writes its hidden state to hidden_out
 * (same layout; it may be the same buffer as hidden_in) and returns no
 * tokens; the last stage returns the greedy tokens (and logits) like
 * pb_prefill_first_token.  Only the stage's layers (and the globals) need to
 * have been streamed: pb_stream_layers accepts a layer_order listing a subset
 * of the layers.  Each layer waits for its own copy, as in a full prefill,
 * and the results are bit-identical to one full prefill.  A stage leaves no
 * decode state.  PB_EINVAL for a bad range or a missing buffer, PB_ESTATE
 * when a needed layer was not streamed. */
int pb_prefill_stage(pb_model* m, const int32_t* tokens, int32_t B, int32_t T, const int32_t* adapter_of_seq,
                     int32_t layer_begin, int32_t layer_end, const float* hidden_in, float* hidden_out,
                     int32_t* out_tokens, float* out_logits);

/* Merged LoRA (Section 4.3.2): fold adapter slot `slot` into the device base
 * weights of every layer, W_t = dt(W_t + scale * B_t A_t) for each of its
 * targets (fp32 product, one rounding), on the compute stream after every
 * layer's copy; blocks until done.  Afterwards the base weights are the merged
 * model: every sequence runs with adapter -1 (a prefill or decode naming any
 * adapter fails with PB_ESTATE) and no LoRA work remains on the hot path.
 * pb_stream_layers (or pb_poison_weights) restores the unmerged state.
 * With merge_shadow, the first merge after a load copies every layer's
 * Wq|Wk|Wv|Wo to the shadow, and a merge while another adapter is merged
 * first restores them from it (an adapter switch: the result is bit-identical
 * to merging onto freshly streamed weights); without, that merge fails with
 * PB_ESTATE.  Requires an attached slot and a prior pb_stream_layers
 * (PB_ESTATE). */
int pb_merge_lora(pb_model* m, int32_t slot);

/* Restore the unmerged base weights from the shadow copy (blocks until done).
 * PB_ESTATE when nothing is merged or the model has no merge_shadow. */
int pb_unmerge_lora(pb_model* m);

/* Epoch-based adapter switching (Section 4.3.2), host side.  Requests are
 * queued per adapter (0 .. n_adapters-1, or -1 for the base model); a batch
 * holds requests of one adapter only, oldest first.  With epoch_batches = E >
 * 0, batches of the active (merged) adapter go first; after E batches of it,
 * or when its queue is empty, the scheduler moves to the other queue whose
 * oldest request has waited longest (staying if no other queue has work).
 * With E = 0 it serves requests in arrival order (the eager baseline: a batch
 * is a run of consecutive arrivals with one adapter).  pb_sched_next reports
 * whether the batch needs another adapter merged than the previous one
 * (`switched`, always 1 for the first batch); the caller merges
 * (pb_merge_lora) or unmerges before running it.  Calls on one scheduler must
 * not overlap. */
typedef struct pb_sched pb_sched;
int pb_sched_create(int32_t n_adapters, int32_t epoch_batches, pb_sched** out);
int pb_sched_destroy(pb_sched* s);
/* PB_EINVAL for an adapter outside [-1, n_adapters). */
int pb_sched_submit(pb_sched* s, int64_t request_id, int32_t adapter);
/* Up to max_batch (>= 1) request ids into ids; *n = 0 when every queue is
 * empty (then *adapter and *switched are left unchanged). */
int pb_sched_next(pb_sched* s, int32_t max_batch, int64_t* ids, int32_t* n, int32_t* adapter,
                  int32_t* switched);
/* Requests still queued, adapter switches so far, the active adapter (-2
 * before the first batch). */
int pb_sched_stats(pb_sched* s, int64_t* pending, int64_t* switches, int32_t* active);

/* KV-cache reconstruction after a failure (Section 4.4.2: a request that was
 * decoding is replayed as one prefill over its prompt and the tokens produced
 * so far).  tokens: host int32 [B*T], sequence-major.  For every layer l with
 * layer_has_kv[l] != 0 the cache still holds keys and values of positions
 * 0..T-1: that layer computes only the queries and attends to the cache; the
 * other layers run a full prefill and store their keys and values.  Returns
 * the next greedy token (and optional logits) of each sequence, like the decode
 * step that would have come next, and leaves the model ready to continue with
 * pb_decode_step.  Requires max_new_tokens > 0 and the prefill's limits. */
int pb_rebuild_kv(pb_model* m, const int32_t* tokens, int32_t B, int32_t T, const int32_t* adapter_of_seq,
                  const uint8_t* layer_has_kv, int32_t* out_tokens, float* out_logits);

/* Overwrite the KV cache of every layer l with layer_lost[l] != 0 with the
 * byte `value` (0xFF: NaN), on the compute stream, and wait for it.  For
 * failure-recovery tests: the cache those layers held is gone, and any read of
 * it before a rebuild shows up as NaN. */
int pb_invalidate_kv(pb_model* m, const uint8_t* layer_lost, int32_t value);

/* Release the model's events and staging (not the caller's arena or streams). */
int pb_destroy(pb_model* m);

/* Thread-local message for the calling thread's last failure ("" if none). */
const char* pb_last_error(void);

/* ---- loader and measurement controls ------------------------------------- */

/* Largest single hipMemcpyAsync the loader issues (default 256 MiB, min 1 MiB). */
int pb_set_chunk_bytes(pb_model* m, size_t bytes);

/* Bytes and elapsed milliseconds (copy-stream events, first copy start to last
 * copy end) of the most recent pb_stream_layers; valid once it has completed. */
int pb_last_load_stats(pb_model* m, double* bytes, double* ms);

/* Graph replay of the forward pass (enabled by default).  Once every weight
 * is resident (the last pb_stream_layers and pb_attach_lora have finished on
 * the device), a forward shape (B, T, prefill or decode step, adapter targets
 * in use) seen a second time is recorded as one HIP graph and replayed on
 * later calls, so the host issues one launch instead of one per kernel.  The
 * recorded kernels and their arguments are those of the launch-by-launch
 * path, so results are bit-identical either way.  A load still in flight,
 * kernel timing or a KV rebuild always runs launch by launch.  Up to 8 shapes
 * are kept per model, least recently used evicted.  enable = 0 turns replay
 * off (recorded graphs are kept for when it is turned on again). */
int pb_set_graph_replay(pb_model* m, int32_t enable);

/* Per-kernel timing of the forward pass.  When enabled, every kernel launch of
 * pb_prefill_first_token is bracketed by events on the compute stream and its
 * duration is added to a per-kernel-kind total (kinds PB_K_*). */
enum {
    PB_K_EMBED = 0, PB_K_LN, PB_K_LORA_SHRINK, PB_K_GEMM_QKV, PB_K_ATTN, PB_K_GEMM_O,
    PB_K_GEMM_FC1, PB_K_GEMM_FC2, PB_K_LM_HEAD, PB_K_ARGMAX, PB_K_COUNT
};
int pb_set_kernel_timing(pb_model* m, int32_t enable);
int pb_get_kernel_timing(pb_model* m, int32_t kind, double* total_ms, int64_t* launches);
int pb_reset_kernel_timing(pb_model* m);

/* Fill the model's device base weights (globals and every layer) with the
 * byte `value` on the copy stream (0xFF makes every weight a NaN), reset the
 * LoRA slots to zeros and mark them empty.  Used to show that no kernel reads
 * a layer before its copy has landed.  Call pb_stream_layers (and
 * pb_attach_lora) again afterwards. */
int pb_poison_weights(pb_model* m, int32_t value);

/* Delay, in microseconds, that the host sleeps between enqueuing consecutive
 * layers in pb_stream_layers (0 = none).  With a delay the compute stream
 * reaches layers whose copies have not been enqueued yet, so a missing wait
 * shows up as NaN from poisoned weights. */
int pb_set_stream_delay_us(pb_model* m, int32_t us);

#ifdef __cplusplus
}
#endif

#endif /* PIPEBOOST_H */
