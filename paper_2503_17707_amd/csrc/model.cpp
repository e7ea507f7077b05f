// Host runtime of the cold-start prefill: layout, loader, forward scheduler
// and the C ABI declared in include/pipeboost.h.
//
// Loading overlaps inference (PipeBoost, Sections 4.2 and 4.3): the loader
// enqueues each layer's host-to-device copies on the copy stream and records
// one event per layer; the forward pass enqueues every layer's kernels on the
// compute stream behind hipStreamWaitEvent(compute, event[layer]).  Waiting
// happens on the device, so the host enqueues the whole forward at once and
// layer l starts the moment its bytes have landed, while later layers are
// still crossing PCIe.  The compute schedule (kernel sequence, tiling,
// reduction orders) never depends on the load order, so results are
// bit-identical for any order.  Once the weights are resident, a repeated forward
// shape is recorded as one HIP graph and replayed (the same launches, no
// per-kernel host work), which matters for warm prefills and decode steps
// whose kernels are short.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cctype>
#include <chrono>
#include <condition_variable>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include <sys/syscall.h>
#include <unistd.h>

#include "../../include/pipeboost.h"
#include "kernels.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

}  // namespace

// The same message slot for the library's other host sources (not exported).
__attribute__((visibility("hidden"))) int pb_fail_status(int code, const char* msg) {
    return fail(code, "%s", msg);
}

namespace {

#define HIP_TRY(call)                                                                  \
    do {                                                                               \
        hipError_t e_ = (call);                                                        \
        if (e_ != hipSuccess)                                                          \
            return fail(PB_EHIP, "%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), \
                        __FILE__, __LINE__);                                           \
    } while (0)

constexpr size_t ALIGN = 256;
constexpr int MAX_SLOTS = 16;
// per-call scalars uploaded in one copy: MAX_SLOTS adapter scales, then the
// position of the first new token
constexpr int SMALL_WORDS = MAX_SLOTS + 1;
// recorded forward passes kept per model (least recently used evicted)
constexpr size_t MAX_GRAPHS = 8;
constexpr int MAX_RANK = 64;
constexpr size_t VEC_ALIGN = 128;  // elements (256 bytes of dt)
// split-K partials: room for 4 fp32 partials of a [max_tokens, d_model]
// output (the o and fc2 projections), between 64 MiB and 1 GiB
size_t gemm_ws_bytes(const pb_config* c) {
    const size_t want = (size_t)4 * c->max_tokens * c->d_model * 4;
    return std::min<size_t>(std::max<size_t>(want, 64u << 20), 1u << 30);
}
constexpr int ROW_SHRINK_MAX_TOKENS = 1024;     // fuse the q/k/v LoRA shrink up to this many tokens
#ifndef PB_COPY_STREAMS
#define PB_COPY_STREAMS 2  // host-to-device copy streams of the loader (1 or 2)
#endif
constexpr int STAGE_SLOTS = 4;                   // pinned staging ring for pageable host blobs
constexpr size_t STAGE_BYTES = 64u << 20;        // ... bytes per slot

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool config_ok(const pb_config* c, std::string* why) {
    auto bad = [&](const char* m) {
        if (why) *why = m;
        return false;
    };
    if (!c) return bad("config is NULL");
    if (c->n_layers < 1) return bad("n_layers must be >= 1");
    if (c->d_model < 128 || c->d_model % 128) return bad("d_model must be a positive multiple of 128");
    if (c->d_model > 16384) return bad("d_model must be <= 16384");
    if (c->n_heads < 1 || c->d_model % c->n_heads) return bad("n_heads must divide d_model");
    const int hd = c->d_model / c->n_heads;
    if (hd != 64 && hd != 128) return bad("head_dim must be 64 or 128");
    if (c->d_ffn < 64 || c->d_ffn % 64) return bad("d_ffn must be a positive multiple of 64");
    if (c->vocab < 1) return bad("vocab must be >= 1");
    if (c->max_pos < 1) return bad("max_pos must be >= 1");
    if (c->max_tokens < 1 || c->max_batch < 1) return bad("max_tokens and max_batch must be >= 1");
    if (c->max_adapters < 0 || c->max_adapters > MAX_SLOTS) return bad("max_adapters must be in [0, 16]");
    if (c->max_adapters > 0 && (c->max_rank < 1 || c->max_rank > MAX_RANK))
        return bad("max_rank must be in [1, 64]");
    if (c->max_new_tokens < 0) return bad("max_new_tokens must be >= 0");
    if (c->merge_shadow != 0 && c->merge_shadow != 1) return bad("merge_shadow must be 0 or 1");
    if (c->dtype != PB_BF16 && c->dtype != PB_F16) return bad("dtype must be PB_BF16 or PB_F16");
    if (!(c->ln_eps > 0.f)) return bad("ln_eps must be > 0");
    return true;
}

struct LayerLayout {
    size_t off[PB_T_COUNT];
    size_t num[PB_T_COUNT];
    size_t total;  // elements
};

LayerLayout layer_layout(const pb_config* c) {
    const size_t d = c->d_model, f = c->d_ffn;
    LayerLayout L{};
    size_t p = 0;
    auto put = [&](int t, size_t n, bool align) {
        if (align) p = align_up(p, VEC_ALIGN);
        L.off[t] = p;
        L.num[t] = n;
        p += n;
    };
    put(PB_T_WQ, d * d, true);
    put(PB_T_WK, d * d, false);
    put(PB_T_WV, d * d, false);
    put(PB_T_WO, d * d, true);
    put(PB_T_W1, f * d, true);
    put(PB_T_W2, d * f, true);
    put(PB_T_BQ, d, true);
    put(PB_T_BK, d, false);
    put(PB_T_BV, d, false);
    put(PB_T_BO, d, true);
    put(PB_T_B1, f, true);
    put(PB_T_B2, d, true);
    put(PB_T_LN1_G, d, true);
    put(PB_T_LN1_B, d, true);
    put(PB_T_LN2_G, d, true);
    put(PB_T_LN2_B, d, true);
    L.total = align_up(p, VEC_ALIGN);
    return L;
}

struct GlobalsLayout {
    size_t off[PB_G_COUNT];
    size_t num[PB_G_COUNT];
    size_t total;
};

GlobalsLayout globals_layout(const pb_config* c) {
    const size_t d = c->d_model;
    GlobalsLayout G{};
    size_t p = 0;
    auto put = [&](int t, size_t n) {
        p = align_up(p, VEC_ALIGN);
        G.off[t] = p;
        G.num[t] = n;
        p += n;
    };
    put(PB_G_EMBED, (size_t)c->vocab * d);
    put(PB_G_POS, (size_t)c->max_pos * d);
    put(PB_G_LNF_G, d);
    put(PB_G_LNF_B, d);
    G.total = align_up(p, VEC_ALIGN);
    return G;
}

int popcount4(uint32_t m) { return (m & 1) + ((m >> 1) & 1) + ((m >> 2) & 1) + ((m >> 3) & 1); }

size_t lora_layer_elems(const pb_config* c, int rank, uint32_t mask) {
    return (size_t)popcount4(mask) * 2 * (size_t)rank * c->d_model;
}

// Everything the arena holds, in bytes.
struct ArenaLayout {
    int rs, kw;  // LoRA slot width (rank rounded up to 8) and packed width (multiple of 64)
    size_t globals, layers, layer_bytes, loraA, loraB, loraA_layer, loraB_layer;
    size_t x, u, qkv, attn, h, z, rowslot, tokens, slotscale, zf, logits, outtok, staging, ws;
    size_t kv, kv_layer, kv_seq;  // KV cache (elements per layer, per sequence)
    size_t shadow, shadow_layer, attn_w;  // unmerged Wq|Wk|Wv|Wo copies: bytes per layer; their offset in a layer
    size_t pval, pidx;
    size_t staging_bytes, ws_bytes, total;
};

ArenaLayout arena_layout(const pb_config* c) {
    ArenaLayout a{};
    const size_t d = c->d_model, f = c->d_ffn, L = c->n_layers, N = c->max_tokens;
    const size_t B = c->max_batch, V = c->vocab;
    a.rs = c->max_adapters > 0 ? (int)align_up(c->max_rank, 8) : 0;
    a.kw = c->max_adapters > 0 ? (int)align_up((size_t)c->max_adapters * a.rs, 64) : 0;
    a.layer_bytes = layer_layout(c).total * 2;
    size_t p = 0;
    auto take = [&](size_t bytes) {
        p = align_up(p, ALIGN);
        const size_t o = p;
        p += bytes;
        return o;
    };
    a.globals = take(globals_layout(c).total * 2);
    a.layers = take(L * a.layer_bytes);
    a.loraA_layer = 4 * (size_t)a.kw * d * 2;
    a.loraB_layer = 4 * d * (size_t)a.kw * 2;
    a.loraA = take(L * a.loraA_layer);
    a.loraB = take(L * a.loraB_layer);
    a.x = take(N * d * 4);
    a.u = take(N * d * 2);
    a.qkv = take(N * 3 * d * 2);
    a.attn = take(N * d * 2);
    a.h = take(N * f * 2);
    a.z = take(N * 4 * (size_t)a.kw * 2);
    a.rowslot = take(N * 4);
    a.tokens = take(N * 4);
    a.slotscale = take(SMALL_WORDS * 4);
    a.zf = take(B * d * 4);
    a.logits = take(B * V * 4);
    a.outtok = take(B * 4);
    a.pval = take(B * (size_t)pb::lm_head_blocks((int)V) * 4);
    a.pidx = take(B * (size_t)pb::lm_head_blocks((int)V) * 4);
    a.staging_bytes = c->max_adapters > 0 ? L * lora_layer_elems(c, c->max_rank, 0xF) * 2 : 0;
    a.staging = take(a.staging_bytes);
    // KV cache for decoding: [L][max_batch][max_pos][k | v] (dt)
    a.kv_seq = c->max_new_tokens > 0 ? (size_t)c->max_pos * 2 * d : 0;
    a.kv_layer = (size_t)B * a.kv_seq;
    a.kv = take(L * a.kv_layer * 2);
    {
        const LayerLayout ll = layer_layout(c);
        a.attn_w = ll.off[PB_T_WQ] * 2;
        a.shadow_layer = c->merge_shadow ? (ll.off[PB_T_WO] + ll.num[PB_T_WO] - ll.off[PB_T_WQ]) * 2 : 0;
        a.shadow = take(L * a.shadow_layer);
    }
    a.ws_bytes = gemm_ws_bytes(c);
    a.ws = take(a.ws_bytes);
    a.total = align_up(p, ALIGN);
    return a;
}

bool is_pinned(const void* p, size_t bytes) {
    if (!p) return false;
    auto one = [](const void* q) {
        hipPointerAttribute_t attr;
        hipError_t e = hipPointerGetAttributes(&attr, q);
        if (e != hipSuccess) {
            (void)hipGetLastError();  // clear the sticky error of the failed query
            return false;
        }
        return attr.type == hipMemoryTypeHost;
    };
    if (!one(p)) return false;
    if (bytes > 1 && !one((const char*)p + bytes - 1)) return false;
    return true;
}

}  // namespace

struct pb_model {
    pb_config cfg;
    ArenaLayout lay;
    LayerLayout ll;
    GlobalsLayout gl;
    char* arena = nullptr;
    hipStream_t copy = nullptr, compute = nullptr;
    // a second copy stream of the library's own: a blob's chunks alternate
    // between the two, so that one copy is queued while the other runs (no
    // idle link between chunks); ev_copy2 joins the second into the first
    hipStream_t copy2 = nullptr;
    hipEvent_t ev_copy2 = nullptr;
    int device = 0;
    std::vector<hipEvent_t> ev_layer;
    hipEvent_t ev_globals = nullptr, ev_lora = nullptr, ev_load0 = nullptr, ev_load1 = nullptr;
    bool streamed = false, lora_recorded = false;
    double last_load_bytes = 0;
    // loader thread (only for loads with pageable blobs): it records each
    // layer's event as that layer's copies are enqueued; `ready` tells the
    // forward pass, on the host, which events exist yet
    std::thread loader;
    std::mutex mu;
    std::condition_variable cv;
    std::vector<char> ready;
    bool globals_ready = false, load_done = true;
    int load_rc = 0;
    std::string load_err;
    char* ring[STAGE_SLOTS] = {};
    hipEvent_t ring_ev[STAGE_SLOTS] = {};
    bool ring_busy[STAGE_SLOTS] = {};
    int ring_next = 0;
    int merged_slot = -1;  // adapter merged into the device base weights (-1: none)
    bool shadow_valid = false;  // the shadow holds this load's unmerged attention weights
    // decode state: sequences of the last prefill, their length so far
    int dec_B = 0, dec_len = 0, dec_steps = 0;
    std::vector<int> dec_adapter;
    size_t chunk_bytes = 256u << 20;
    int delay_us = 0;
    // adapter slots
    bool slot_valid[MAX_SLOTS] = {};
    int slot_rank[MAX_SLOTS] = {};
    uint32_t slot_mask[MAX_SLOTS] = {};
    float slot_scale[MAX_SLOTS] = {};
    // pinned host staging for the small per-call transfers
    int32_t* h_tokens = nullptr;
    int32_t* h_rowslot = nullptr;
    float* h_scale = nullptr;
    int32_t* h_outtok = nullptr;
    float* h_logits = nullptr;
    // recorded forward passes, replayed once the weights have settled; an
    // entry with no exec has been seen once (a shape seen once is not recorded)
    struct Graph {
        int B, T;
        bool decode, use_lora;
        uint32_t lora_union;
        hipGraphExec_t exec;
        uint64_t last_use;
    };
    std::vector<Graph> graphs;
    uint64_t graph_clock = 0;
    bool graphs_on = true;
    // per-kernel timing
    bool timing = false;
    std::vector<hipEvent_t> tev;
    std::vector<int> tkind;
    size_t tused = 0;
    double ttotal[PB_K_COUNT] = {};
    int64_t tcount[PB_K_COUNT] = {};

    char* at(size_t off) { return arena + off; }
    char* layer_ptr(int l) { return at(lay.layers + (size_t)l * lay.layer_bytes); }
    char* ltensor(int l, int t) { return layer_ptr(l) + ll.off[t] * 2; }
    char* gtensor(int t) { return at(lay.globals) + gl.off[t] * 2; }
};

extern "C" {

const char* pb_last_error(void) { return g_err.c_str(); }

size_t pb_layer_bytes(const pb_config* cfg) {
    if (!config_ok(cfg, nullptr)) return 0;
    return layer_layout(cfg).total * 2;
}

size_t pb_globals_bytes(const pb_config* cfg) {
    if (!config_ok(cfg, nullptr)) return 0;
    return globals_layout(cfg).total * 2;
}

int pb_layer_tensor(const pb_config* cfg, int32_t tensor, size_t* offset, size_t* numel) {
    std::string why;
    if (!config_ok(cfg, &why)) return fail(PB_EINVAL, "invalid config: %s", why.c_str());
    if (tensor < 0 || tensor >= PB_T_COUNT) return fail(PB_EINVAL, "unknown layer tensor %d", tensor);
    const LayerLayout L = layer_layout(cfg);
    if (offset) *offset = L.off[tensor];
    if (numel) *numel = L.num[tensor];
    return PB_OK;
}

int pb_globals_tensor(const pb_config* cfg, int32_t tensor, size_t* offset, size_t* numel) {
    std::string why;
    if (!config_ok(cfg, &why)) return fail(PB_EINVAL, "invalid config: %s", why.c_str());
    if (tensor < 0 || tensor >= PB_G_COUNT) return fail(PB_EINVAL, "unknown global tensor %d", tensor);
    const GlobalsLayout G = globals_layout(cfg);
    if (offset) *offset = G.off[tensor];
    if (numel) *numel = G.num[tensor];
    return PB_OK;
}

size_t pb_lora_layer_bytes(const pb_config* cfg, int32_t rank, uint32_t target_mask) {
    if (!config_ok(cfg, nullptr) || rank < 1 || rank > cfg->max_rank || (target_mask & ~0xFu) ||
        target_mask == 0)
        return 0;
    return lora_layer_elems(cfg, rank, target_mask) * 2;
}

int pb_lora_tensor(const pb_config* cfg, int32_t rank, uint32_t target_mask, int32_t target,
                   int32_t which, size_t* offset, size_t* numel) {
    if (pb_lora_layer_bytes(cfg, rank, target_mask) == 0)
        return fail(PB_EINVAL, "invalid LoRA rank %d or target mask 0x%x", rank, target_mask);
    if (target < 0 || target > 3 || !((target_mask >> target) & 1u))
        return fail(PB_EINVAL, "target %d not in mask 0x%x", target, target_mask);
    if (which != 0 && which != 1) return fail(PB_EINVAL, "which must be 0 (A) or 1 (B)");
    int idx = 0;
    for (int t = 0; t < target; ++t) idx += (target_mask >> t) & 1u;
    const size_t rd = (size_t)rank * cfg->d_model;
    if (offset) *offset = (size_t)idx * 2 * rd + (which ? rd : 0);
    if (numel) *numel = rd;
    return PB_OK;
}

size_t pb_arena_bytes(const pb_config* cfg) {
    if (!config_ok(cfg, nullptr)) return 0;
    return arena_layout(cfg).total;
}

namespace {

// NUMA node that pinned allocations are placed on (-1: the runtime's choice)
std::atomic<int> g_host_node{-1};

// MPOL_PREFERRED of one node for the calling thread while it lives, so that
// hipHostMalloc with hipHostMallocNumaUser takes its pages there (other
// nodes only if that one is full); the default policy is restored afterwards
struct BindThreadToNode {
    bool active = false;
    explicit BindThreadToNode(int node) {
        if (node < 0 || node >= 1024) return;
        unsigned long mask[1024 / (8 * sizeof(unsigned long))] = {};
        mask[node / (8 * sizeof(unsigned long))] = 1UL << (node % (8 * sizeof(unsigned long)));
        active = syscall(SYS_set_mempolicy, 1 /* MPOL_PREFERRED */, mask, (unsigned long)1024) == 0;
    }
    ~BindThreadToNode() {
        if (active) (void)syscall(SYS_set_mempolicy, 0 /* MPOL_DEFAULT */, nullptr, 0UL);
    }
};

hipError_t host_malloc_on_node(void** out, size_t bytes) {
    const int node = g_host_node.load();
    if (node < 0) return hipHostMalloc(out, bytes, hipHostMallocDefault);
    BindThreadToNode bind(node);
    return hipHostMalloc(out, bytes, bind.active ? hipHostMallocNumaUser : hipHostMallocDefault);
}

}  // namespace

int pb_host_numa_node(int32_t device, int32_t* node) {
    if (!node) return fail(PB_EINVAL, "pb_host_numa_node: node is NULL");
    *node = -1;
    char bus[64] = {};
    HIP_TRY(hipDeviceGetPCIBusId(bus, (int)sizeof(bus) - 1, device));
    for (char* c = bus; *c; ++c) *c = (char)std::tolower((unsigned char)*c);
    const std::string path = std::string("/sys/bus/pci/devices/") + bus + "/numa_node";
    FILE* f = std::fopen(path.c_str(), "r");
    if (!f) return PB_OK;  // no NUMA information: -1
    int v = -1;
    if (std::fscanf(f, "%d", &v) != 1) v = -1;
    std::fclose(f);
    *node = v;
    return PB_OK;
}

int pb_set_host_numa_node(int32_t node) {
    if (node < -1 || node >= 1024) return fail(PB_EINVAL, "pb_set_host_numa_node: node %d out of range", node);
    g_host_node.store(node);
    return PB_OK;
}

int pb_host_alloc(size_t bytes, void** out) {
    if (!out || bytes == 0) return fail(PB_EINVAL, "pb_host_alloc: bad arguments");
    *out = nullptr;
    hipError_t e = host_malloc_on_node(out, bytes);
    if (e != hipSuccess) {
        *out = nullptr;
        return fail(PB_ENOMEM, "hipHostMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
    }
    return PB_OK;
}

int pb_host_free(void* ptr) {
    if (!ptr) return PB_OK;
    HIP_TRY(hipHostFree(ptr));
    return PB_OK;
}

int pb_model_create(const pb_config* cfg, void* dev_arena, size_t arena_bytes, void* copy_stream,
                    void* compute_stream, pb_model** out) {
    if (!out) return fail(PB_EINVAL, "out is NULL");
    *out = nullptr;
    std::string why;
    if (!config_ok(cfg, &why)) return fail(PB_EINVAL, "invalid config: %s", why.c_str());
    if (!dev_arena || ((uintptr_t)dev_arena % ALIGN))
        return fail(PB_EINVAL, "device arena must be non-NULL and 256-byte aligned");
    if (copy_stream == compute_stream)
        return fail(PB_EINVAL, "copy and compute streams must differ");
    const ArenaLayout lay = arena_layout(cfg);
    if (arena_bytes < lay.total)
        return fail(PB_ENOMEM, "arena of %zu bytes is smaller than the %zu required", arena_bytes,
                    lay.total);
    pb_model* m = new pb_model();
    m->cfg = *cfg;
    m->lay = lay;
    m->ll = layer_layout(cfg);
    m->gl = globals_layout(cfg);
    m->arena = (char*)dev_arena;
    m->copy = (hipStream_t)copy_stream;
    m->compute = (hipStream_t)compute_stream;
    auto cleanup = [&](int code) {
        pb_destroy(m);
        return code;
    };
    if (hipGetDevice(&m->device) != hipSuccess) return cleanup(fail(PB_EHIP, "hipGetDevice failed"));
    m->ev_layer.assign(cfg->n_layers, nullptr);
    for (auto& e : m->ev_layer)
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess)
            return cleanup(fail(PB_EHIP, "hipEventCreate failed"));
    if (PB_COPY_STREAMS > 1 &&
        (hipStreamCreateWithFlags(&m->copy2, hipStreamNonBlocking) != hipSuccess ||
         hipEventCreateWithFlags(&m->ev_copy2, hipEventDisableTiming) != hipSuccess))
        return cleanup(fail(PB_EHIP, "second copy stream creation failed"));
    if (hipEventCreateWithFlags(&m->ev_globals, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&m->ev_lora, hipEventDisableTiming) != hipSuccess ||
        hipEventCreate(&m->ev_load0) != hipSuccess || hipEventCreate(&m->ev_load1) != hipSuccess)
        return cleanup(fail(PB_EHIP, "hipEventCreate failed"));
    const size_t B = cfg->max_batch, N = cfg->max_tokens, V = cfg->vocab;
    if (hipHostMalloc((void**)&m->h_tokens, N * 4, 0) != hipSuccess ||
        hipHostMalloc((void**)&m->h_rowslot, N * 4, 0) != hipSuccess ||
        hipHostMalloc((void**)&m->h_scale, SMALL_WORDS * 4, 0) != hipSuccess ||
        hipHostMalloc((void**)&m->h_outtok, B * 4, 0) != hipSuccess ||
        hipHostMalloc((void**)&m->h_logits, B * V * 4, 0) != hipSuccess)
        return cleanup(fail(PB_ENOMEM, "pinned staging allocation failed"));
    // LoRA slots start as zeros: an empty slot contributes exactly nothing
    {
        const size_t end = lay.loraB + (size_t)cfg->n_layers * lay.loraB_layer;
        if (end > lay.loraA && hipMemsetAsync(m->at(lay.loraA), 0, end - lay.loraA, m->copy) != hipSuccess)
            return cleanup(fail(PB_EHIP, "hipMemsetAsync of the LoRA slots failed"));
    }
    if (hipStreamSynchronize(m->copy) != hipSuccess)
        return cleanup(fail(PB_EHIP, "hipStreamSynchronize failed"));
    *out = m;
    return PB_OK;
}

int pb_destroy(pb_model* m) {
    if (!m) return PB_OK;
    if (m->loader.joinable()) m->loader.join();
    if (m->copy) (void)hipStreamSynchronize(m->copy);
    if (m->copy2) (void)hipStreamSynchronize(m->copy2);
    if (m->compute) (void)hipStreamSynchronize(m->compute);
    for (auto e : m->ev_layer)
        if (e) (void)hipEventDestroy(e);
    for (auto e : m->tev)
        if (e) (void)hipEventDestroy(e);
    for (auto e : {m->ev_globals, m->ev_lora, m->ev_load0, m->ev_load1})
        if (e) (void)hipEventDestroy(e);
    for (auto& g : m->graphs)
        if (g.exec) (void)hipGraphExecDestroy(g.exec);
    for (void* p : {(void*)m->h_tokens, (void*)m->h_rowslot, (void*)m->h_scale, (void*)m->h_outtok,
                    (void*)m->h_logits})
        if (p) (void)hipHostFree(p);
    for (int k = 0; k < STAGE_SLOTS; ++k) {
        if (m->ring[k]) (void)hipHostFree(m->ring[k]);
        if (m->ring_ev[k]) (void)hipEventDestroy(m->ring_ev[k]);
    }
    if (m->ev_copy2) (void)hipEventDestroy(m->ev_copy2);
    if (m->copy2) (void)hipStreamDestroy(m->copy2);
    delete m;
    return PB_OK;
}

int pb_set_chunk_bytes(pb_model* m, size_t bytes) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    if (bytes < (1u << 20)) return fail(PB_EINVAL, "chunk must be at least 1 MiB");
    m->chunk_bytes = bytes;
    return PB_OK;
}

int pb_set_stream_delay_us(pb_model* m, int32_t us) {
    if (!m || us < 0) return fail(PB_EINVAL, "bad arguments");
    m->delay_us = us;
    return PB_OK;
}

// Copy stream of chunk i of a blob: the chunks alternate between the two
// copy streams (when there are two); join_copy2 then makes the first stream
// wait for the second, so an event recorded on the first covers the blob.
static hipStream_t chunk_stream(pb_model* m, size_t i) { return (m->copy2 && (i & 1)) ? m->copy2 : m->copy; }

static int join_copy2(pb_model* m, size_t chunks) {
    if (!m->copy2 || chunks < 2) return PB_OK;
    HIP_TRY(hipEventRecord(m->ev_copy2, m->copy2));
    HIP_TRY(hipStreamWaitEvent(m->copy, m->ev_copy2, 0));
    return PB_OK;
}

static int copy_chunked(pb_model* m, char* dst, const char* src, size_t bytes) {
    // with two streams a blob goes in at least two chunks
    size_t chunk = m->chunk_bytes;
    if (m->copy2 && bytes > 2 * (1u << 20)) chunk = std::min(chunk, ((bytes + 1) / 2 + 4095) & ~(size_t)4095);
    size_t i = 0;
    for (size_t o = 0; o < bytes; o += chunk, ++i) {
        const size_t n = std::min(chunk, bytes - o);
        HIP_TRY(hipMemcpyAsync(dst + o, src + o, n, hipMemcpyHostToDevice, chunk_stream(m, i)));
    }
    return join_copy2(m, i);
}

// Host copy split over several threads (pageable source -> pinned ring slot).
static void parallel_memcpy(char* dst, const char* src, size_t n) {
    const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
    const size_t parts = std::min<size_t>(std::min(8u, hw), std::max<size_t>(1, n >> 22));
    const size_t step = ((n + parts - 1) / parts + 4095) & ~(size_t)4095;
    std::vector<std::thread> pool;
    for (size_t i = 1; i < parts && i * step < n; ++i)
        pool.emplace_back([=] { std::memcpy(dst + i * step, src + i * step, std::min(step, n - i * step)); });
    std::memcpy(dst, src, std::min(step, n));
    for (auto& t : pool) t.join();
}

// A pageable blob: through the pinned ring, each slot reused once its DMA
// (an event on the copy stream) has finished.
static int copy_staged(pb_model* m, char* dst, const char* src, size_t bytes) {
    size_t i = 0;
    for (size_t o = 0; o < bytes; o += STAGE_BYTES, ++i) {
        const size_t n = std::min(STAGE_BYTES, bytes - o);
        const int k = m->ring_next;
        m->ring_next = (k + 1) % STAGE_SLOTS;
        if (m->ring_busy[k]) HIP_TRY(hipEventSynchronize(m->ring_ev[k]));
        parallel_memcpy(m->ring[k], src + o, n);
        const hipStream_t cs = chunk_stream(m, i);
        HIP_TRY(hipMemcpyAsync(dst + o, m->ring[k], n, hipMemcpyHostToDevice, cs));
        HIP_TRY(hipEventRecord(m->ring_ev[k], cs));
        m->ring_busy[k] = true;
    }
    return join_copy2(m, i);
}

struct LoadJob {
    const char* src;
    char* dst;
    size_t bytes;
    bool pinned;
    int layer;  // -1 = globals
};

// Enqueue every blob in order, recording the per-layer events; marks each
// event as recorded for the forward pass.  Returns the first failure.
static int run_load(pb_model* m, const std::vector<LoadJob>& jobs) {
    for (size_t i = 0; i < jobs.size(); ++i) {
        const LoadJob& j = jobs[i];
        if (m->delay_us > 0 && i > 1) std::this_thread::sleep_for(std::chrono::microseconds(m->delay_us));
        const int rc = j.pinned ? copy_chunked(m, j.dst, j.src, j.bytes) : copy_staged(m, j.dst, j.src, j.bytes);
        if (rc) return rc;
        HIP_TRY(hipEventRecord(j.layer < 0 ? m->ev_globals : m->ev_layer[j.layer], m->copy));
        {
            std::lock_guard<std::mutex> lk(m->mu);
            if (j.layer < 0) m->globals_ready = true;
            else m->ready[j.layer] = 1;
        }
        m->cv.notify_all();
    }
    HIP_TRY(hipEventRecord(m->ev_load1, m->copy));
    return PB_OK;
}

static void finish_load(pb_model* m, int rc) {
    {
        std::lock_guard<std::mutex> lk(m->mu);
        m->load_rc = rc;
        m->load_err = rc ? g_err : std::string();
        m->load_done = true;
    }
    m->cv.notify_all();
}

// Wait (on the host) until the event of `layer` (-1: globals) has been
// recorded by the current load.
static int wait_recorded(pb_model* m, int layer) {
    std::unique_lock<std::mutex> lk(m->mu);
    auto have = [&] { return layer < 0 ? m->globals_ready : m->ready[layer] != 0; };
    m->cv.wait(lk, [&] { return have() || m->load_done; });
    if (have()) return PB_OK;
    return fail(m->load_rc ? m->load_rc : PB_ESTATE, "layer %d was not loaded: %s", layer, m->load_err.c_str());
}

// Join a previous load's thread; its failure, if any, is reported here.
static int join_load(pb_model* m) {
    if (m->loader.joinable()) m->loader.join();
    if (m->load_rc) return fail(m->load_rc, "%s", m->load_err.c_str());
    return PB_OK;
}

int pb_stream_layers(pb_model* m, const int32_t* layer_order, int32_t n_layers,
                     const void* const* host_layers, const void* host_globals) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    if (m->loader.joinable()) m->loader.join();
    m->load_rc = 0;
    const int L = m->cfg.n_layers;
    if (n_layers < 1 || n_layers > L)
        return fail(PB_EINVAL, "layer_order has %d entries, the model %d layers", n_layers, L);
    if (!layer_order || !host_layers || !host_globals) return fail(PB_EINVAL, "NULL argument");
    std::vector<char> seen(L, 0);
    for (int i = 0; i < n_layers; ++i) {
        const int l = layer_order[i];
        if (l < 0 || l >= L || seen[l]) return fail(PB_EINVAL, "layer_order entry %d is out of range or repeated", l);
        seen[l] = 1;
        if (!host_layers[l]) return fail(PB_EINVAL, "layer %d blob is NULL", l);
    }
    const size_t lb = m->lay.layer_bytes, gb = m->gl.total * 2;
    std::vector<LoadJob> jobs;
    jobs.push_back({(const char*)host_globals, m->at(m->lay.globals), gb, is_pinned(host_globals, gb), -1});
    for (int i = 0; i < n_layers; ++i) {
        const int l = layer_order[i];
        jobs.push_back({(const char*)host_layers[l], m->layer_ptr(l), lb, is_pinned(host_layers[l], lb), l});
    }
    const bool all_pinned = std::all_of(jobs.begin(), jobs.end(), [](const LoadJob& j) { return j.pinned; });
    if (!all_pinned && !m->ring[0]) {
        for (int k = 0; k < STAGE_SLOTS; ++k) {
            if (host_malloc_on_node((void**)&m->ring[k], STAGE_BYTES) != hipSuccess)
                return fail(PB_ENOMEM, "pinned staging ring allocation failed");
            HIP_TRY(hipEventCreateWithFlags(&m->ring_ev[k], hipEventDisableTiming));
        }
    }
    {
        std::lock_guard<std::mutex> lk(m->mu);
        m->ready.assign(L, 0);
        m->globals_ready = false;
        m->load_done = false;
        m->load_err.clear();
    }
    HIP_TRY(hipEventRecord(m->ev_load0, m->copy));
    // the second copy stream starts after everything enqueued on the first
    // (the weight poisoning of a cold-start measurement, earlier loads)
    if (m->copy2) HIP_TRY(hipStreamWaitEvent(m->copy2, m->ev_load0, 0));
    m->last_load_bytes = (double)gb + (double)n_layers * (double)lb;
    m->merged_slot = -1;  // the base weights arrive unmerged
    m->shadow_valid = false;
    if (all_pinned) {
        // every copy is a DMA from locked pages: enqueue them all now
        const int rc = run_load(m, jobs);
        finish_load(m, rc);
        if (rc) return rc;
        m->streamed = true;
        return PB_OK;
    }
    // pageable blobs need host copies into the ring: a loader thread enqueues
    // the copies in order while this call returns (the forward pass waits on
    // the host for each layer's event to exist)
    m->streamed = true;
    m->loader = std::thread([m, jobs = std::move(jobs)] {
        int rc = hipSetDevice(m->device) == hipSuccess ? PB_OK : fail(PB_EHIP, "hipSetDevice failed");
        if (!rc) rc = run_load(m, jobs);
        finish_load(m, rc);
    });
    return PB_OK;
}

int pb_attach_lora(pb_model* m, int32_t slot, int32_t rank, float alpha, uint32_t target_mask,
                   const void* const* host_lora) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    if (m->loader.joinable()) m->loader.join();  // the copy stream's order stays the caller's
    const pb_config& c = m->cfg;
    if (slot < 0 || slot >= c.max_adapters) return fail(PB_EINVAL, "slot %d outside [0, %d)", slot, c.max_adapters);
    if (rank < 1 || rank > c.max_rank) return fail(PB_EINVAL, "rank %d outside [1, %d]", rank, c.max_rank);
    if (target_mask == 0 || (target_mask & ~0xFu)) return fail(PB_EINVAL, "bad target mask 0x%x", target_mask);
    if (!std::isfinite(alpha)) return fail(PB_EINVAL, "alpha must be finite");
    if (!host_lora) return fail(PB_EINVAL, "host_lora is NULL");
    const size_t elems = lora_layer_elems(&c, rank, target_mask);
    const size_t bytes = elems * 2;
    for (int l = 0; l < c.n_layers; ++l)
        if (!is_pinned(host_lora[l], bytes)) return fail(PB_ENOTPINNED, "LoRA blob of layer %d is not pinned", l);
    char* stage = m->at(m->lay.staging);
    for (int l = 0; l < c.n_layers; ++l)
        HIP_TRY(hipMemcpyAsync(stage + (size_t)l * bytes, host_lora[l], bytes, hipMemcpyHostToDevice, m->copy));
    HIP_TRY(pb::launch_lora_pack(c.dtype, stage, elems, c.n_layers, c.d_model, rank, target_mask, slot,
                                 m->lay.rs, m->lay.kw, m->at(m->lay.loraA), m->at(m->lay.loraB),
                                 m->copy));
    HIP_TRY(hipEventRecord(m->ev_lora, m->copy));
    m->lora_recorded = true;
    m->slot_valid[slot] = true;
    m->slot_rank[slot] = rank;
    m->slot_mask[slot] = target_mask;
    m->slot_scale[slot] = alpha / (float)rank;
    return PB_OK;
}

int pb_poison_weights(pb_model* m, int32_t value) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    if (m->loader.joinable()) m->loader.join();
    const ArenaLayout& a = m->lay;
    HIP_TRY(hipMemsetAsync(m->at(a.globals), value & 0xFF, a.loraA - a.globals, m->copy));
    // LoRA slots go back to zeros (a NaN in an unused slot would reach every
    // output through the zero columns of the packed expand); they hold no
    // adapter until the next pb_attach_lora
    const size_t end = a.loraB + (size_t)m->cfg.n_layers * a.loraB_layer;
    if (end > a.loraA) HIP_TRY(hipMemsetAsync(m->at(a.loraA), 0, end - a.loraA, m->copy));
    for (int s = 0; s < MAX_SLOTS; ++s) m->slot_valid[s] = false;
    m->streamed = false;
    m->dec_B = 0;
    m->merged_slot = -1;
    m->shadow_valid = false;
    return PB_OK;
}

int pb_last_load_stats(pb_model* m, double* bytes, double* ms) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    if (!m->streamed) return fail(PB_ESTATE, "no completed pb_stream_layers");
    if (int rc = join_load(m)) return rc;
    float t = 0.f;
    HIP_TRY(hipEventSynchronize(m->ev_load1));
    HIP_TRY(hipEventElapsedTime(&t, m->ev_load0, m->ev_load1));
    if (bytes) *bytes = m->last_load_bytes;
    if (ms) *ms = t;
    return PB_OK;
}

int pb_set_graph_replay(pb_model* m, int32_t enable) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    m->graphs_on = enable != 0;
    return PB_OK;
}

int pb_set_kernel_timing(pb_model* m, int32_t enable) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    m->timing = enable != 0;
    return PB_OK;
}

int pb_get_kernel_timing(pb_model* m, int32_t kind, double* total_ms, int64_t* launches) {
    if (!m || kind < 0 || kind >= PB_K_COUNT) return fail(PB_EINVAL, "bad arguments");
    if (total_ms) *total_ms = m->ttotal[kind];
    if (launches) *launches = m->tcount[kind];
    return PB_OK;
}

int pb_reset_kernel_timing(pb_model* m) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    for (int k = 0; k < PB_K_COUNT; ++k) {
        m->ttotal[k] = 0;
        m->tcount[k] = 0;
    }
    return PB_OK;
}

}  // extern "C"

namespace {

// Times the launches of one kernel kind (a GEMM and its split-K reduce, say)
// when timing is enabled: the events come from the kernels' own dispatch
// packets (the first launch's start, the last one's end), so the span holds
// no marker packets of its own.
struct Timed {
    pb_model* m;
    int kind;
    size_t idx;
    Timed(pb_model* mm, int k) : m(mm), kind(k), idx(0) {
        if (!m->timing) return;
        if (m->tused + 2 > m->tev.size()) {
            hipEvent_t a, b;
            (void)hipEventCreate(&a);
            (void)hipEventCreate(&b);
            m->tev.push_back(a);
            m->tev.push_back(b);
            m->tkind.push_back(-1);
        }
        idx = m->tused;
        m->tused += 2;
        m->tkind[idx / 2] = kind;
        pb::g_launch_timing = {m->tev[idx], m->tev[idx + 1]};
    }
    ~Timed() {
        if (!m->timing) return;
        if (pb::g_launch_timing.start) {  // nothing was launched: an empty span
            (void)hipEventRecord(m->tev[idx], m->compute);
            (void)hipEventRecord(m->tev[idx + 1], m->compute);
        }
        pb::g_launch_timing = {nullptr, nullptr};
    }
};

// The forward pass of B sequences of T new tokens at positions pos0 ..
// pos0+T-1, pos0 read from device memory.  A prefill (decode = false) attends
// among its own tokens; a decode step (T = 1) attends to the KV cache, which
// both append to when the model keeps one.  With wait_loads the compute
// stream waits for each layer's copy event before the layer's first kernel
// (the pipelined cold start); without, every weight must already be resident
// (a recorded pass holds no waits on the load's events).
// One pipeline stage's share of the forward pass: layers [l0, l1), the
// hidden state (fp32 [N, d], device) taken from `in` unless the stage starts
// at layer 0 (embedding) and handed to `out` unless it ends at the last layer
// (final LayerNorm, LM head, argmax).
struct Stage {
    int l0, l1;
    const float* in;
    float* out;
};

int enqueue_forward(pb_model* m, int B, int T, bool use_lora, uint32_t lora_union, bool decode,
                    const uint8_t* has_kv, bool wait_loads, const Stage* st = nullptr) {
    const pb_config& c = m->cfg;
    const ArenaLayout& a = m->lay;
    const int dt = c.dtype;
    const int d = c.d_model, F = c.d_ffn, H = c.n_heads, hd = d / H, L = c.n_layers;
    const int N = B * T;
    hipStream_t s = m->compute;
    float* x = (float*)m->at(a.x);
    char* u = m->at(a.u);
    char* qkv = m->at(a.qkv);
    char* attn = m->at(a.attn);
    char* hbuf = m->at(a.h);
    char* z = m->at(a.z);
    const int kw = a.kw;
    const int32_t* rowslot = (const int32_t*)m->at(a.rowslot);
    const float* sscale = (const float*)m->at(a.slotscale);
    const pb::GemmWorkspace gws{m->at(a.ws), a.ws_bytes};
    const int32_t* pos0 = (const int32_t*)(m->at(a.slotscale) + MAX_SLOTS * 4);
    auto wait_layer = [&](int l) -> int {
        if (!wait_loads) return PB_OK;
        if (int rc = wait_recorded(m, l)) return rc;
        HIP_TRY(hipStreamWaitEvent(s, l < 0 ? m->ev_globals : m->ev_layer[l], 0));
        return PB_OK;
    };

    const int l0 = st ? st->l0 : 0, l1 = st ? st->l1 : L;
    if (int rc = wait_layer(-1)) return rc;
    if (use_lora && wait_loads) HIP_TRY(hipStreamWaitEvent(s, m->ev_lora, 0));
    if (l0 == 0) {
        Timed t(m, PB_K_EMBED);
        HIP_TRY(pb::launch_embed(dt, (const int32_t*)m->at(a.tokens), m->gtensor(PB_G_EMBED),
                                 m->gtensor(PB_G_POS), x, N, T, d, pos0, s));
    } else {  // the previous stage's hidden state
        HIP_TRY(hipMemcpyAsync(x, st->in, (size_t)N * d * 4, hipMemcpyDeviceToDevice, s));
    }
    const bool qkv_lora = use_lora && (lora_union & (PB_LORA_Q | PB_LORA_K | PB_LORA_V));
    const bool o_lora = use_lora && (lora_union & PB_LORA_O);
    // Up to 1024 tokens the q/k/v LoRA shrink rides on the kernel that writes
    // the LayerNorm rows (row-wise dot products; for a handful of rows, decode
    // steps, each row's 16-rank groups go to blocks of their own so that the A
    // reads spread over several CUs); for more tokens it is a GEMM.
    const bool fuse_shrink = qkv_lora && N <= ROW_SHRINK_MAX_TOKENS;
    auto row_shrink_args = [&](int layer) {
        pb::RowShrink sh{};
        if (fuse_shrink) {
            sh.Acat = m->at(a.loraA) + (size_t)layer * a.loraA_layer;
            sh.row_slot = rowslot; sh.slot_scale = sscale; sh.Z = z;
            sh.rs = a.rs; sh.kw = kw; sh.mask = lora_union & 7u;
        }
        return sh;
    };
    bool ln1_ready = false;  // LN1 (and its fused shrink) of layer l produced by layer l-1's fc2 reduce
    for (int l = l0; l < l1; ++l) {
        if (int rc = wait_layer(l)) return rc;
        char* Aq = m->at(a.loraA) + (size_t)l * a.loraA_layer;  // [4][kw][d]
        char* Bq = m->at(a.loraB) + (size_t)l * a.loraB_layer;  // [4][d][kw]
        if (!ln1_ready) {
            Timed t(m, PB_K_LN);
            const pb::RowShrink sh = row_shrink_args(l);
            HIP_TRY(pb::launch_layernorm(dt, x, 1, 0, m->ltensor(l, PB_T_LN1_G), m->ltensor(l, PB_T_LN1_B),
                                         u, false, N, d, c.ln_eps, s, &sh));
        }
        ln1_ready = false;
        if (qkv_lora && !fuse_shrink) {
            Timed t(m, PB_K_LORA_SHRINK);
            pb::GemmParams p{};
            p.X = u; p.ldx = d; p.W = Aq; p.ldw = d; p.M = N; p.N = 3 * kw; p.K1 = d;
            p.C = z; p.ldc = 4 * kw;
            p.row_slot = rowslot; p.slot_scale = sscale; p.slot_width = a.rs; p.kw = kw;
            HIP_TRY(pb::launch_gemm(dt, 4, pb::EPI_SHRINK, p, gws, s));
        }
        // a layer whose cache already holds keys and values for every position
        // (KV rebuild) computes only the queries and attends to the cache
        const bool reuse_kv = has_kv && has_kv[l];
        {
            Timed t(m, PB_K_GEMM_QKV);
            pb::GemmParams p{};
            p.X = u; p.ldx = d; p.W = m->ltensor(l, PB_T_WQ); p.ldw = d; p.M = N; p.N = (reuse_kv ? 1 : 3) * d;
            p.K1 = d;
            if (qkv_lora && (!reuse_kv || (lora_union & PB_LORA_Q))) {
                p.X2 = z; p.ldx2 = 4 * kw; p.W2 = Bq; p.ldw2 = kw; p.K2 = kw; p.group = d;
                p.k2_mask = lora_union & (reuse_kv ? 1u : 7u); p.x2_group_stride = kw;
            }
            p.bias = m->ltensor(l, PB_T_BQ);
            p.C = qkv; p.ldc = 3 * d;
            p.qscale = 1.0f / std::sqrt((float)hd); p.qcols = d;
            if (a.kv_layer && !reuse_kv) {  // keys and values of the new tokens into the cache
                p.kv = m->at(a.kv) + (size_t)l * a.kv_layer * 2;
                p.kv_pos = pos0; p.kv_T = T; p.kv_seq = (int64_t)a.kv_seq;
            }
            HIP_TRY(pb::launch_gemm(dt, 0, pb::EPI_QKV, p, gws, s));
        }
        {
            Timed t(m, PB_K_ATTN);
            if (reuse_kv) {
                const char* kvl = m->at(a.kv) + (size_t)l * a.kv_layer * 2;
                HIP_TRY(pb::launch_attention_kv(dt, qkv, kvl, 2 * (int64_t)d, (int64_t)a.kv_seq, attn, B, T, H,
                                                hd, s));
            } else if (!decode) {
                HIP_TRY(pb::launch_attention(dt, qkv, attn, B, T, H, hd, s));
            } else {
                const char* kvl = m->at(a.kv) + (size_t)l * a.kv_layer * 2;
                HIP_TRY(pb::launch_decode_attention(dt, qkv, kvl, (int64_t)a.kv_seq, B, H, hd, pos0, attn, s));
            }
        }
        if (o_lora) {
            Timed t(m, PB_K_LORA_SHRINK);
            pb::GemmParams p{};
            p.X = attn; p.ldx = d; p.W = Aq + 3 * (size_t)kw * d * 2; p.ldw = d; p.M = N; p.N = kw; p.K1 = d;
            p.C = z + 3 * (size_t)kw * 2; p.ldc = 4 * kw;
            p.row_slot = rowslot; p.slot_scale = sscale; p.slot_width = a.rs; p.kw = kw;
            HIP_TRY(pb::launch_gemm(dt, 4, pb::EPI_SHRINK, p, gws, s));
        }
        bool ln2_done = false;
        {
            Timed t(m, PB_K_GEMM_O);
            pb::GemmParams p{};
            p.X = attn; p.ldx = d; p.W = m->ltensor(l, PB_T_WO); p.ldw = d; p.M = N; p.N = d; p.K1 = d;
            if (o_lora) {
                p.X2 = z + 3 * (size_t)kw * 2; p.ldx2 = 4 * kw; p.W2 = Bq + 3 * (size_t)d * kw * 2;
                p.ldw2 = kw; p.K2 = kw; p.group = d; p.k2_mask = 1u; p.x2_group_stride = 0;
            }
            p.bias = m->ltensor(l, PB_T_BO);
            p.R = x; p.ldr = d;
            // LN2 rides on the split-K reduce when the launcher splits
            p.ln_g = m->ltensor(l, PB_T_LN2_G); p.ln_b = m->ltensor(l, PB_T_LN2_B); p.ln_out = u;
            p.ln_eps = c.ln_eps; p.ln_done = &ln2_done;
            HIP_TRY(pb::launch_gemm(dt, 1, pb::EPI_RESID, p, gws, s));
        }
        if (!ln2_done) {
            Timed t(m, PB_K_LN);
            HIP_TRY(pb::launch_layernorm(dt, x, 1, 0, m->ltensor(l, PB_T_LN2_G), m->ltensor(l, PB_T_LN2_B),
                                         u, false, N, d, c.ln_eps, s));
        }
        {
            Timed t(m, PB_K_GEMM_FC1);
            pb::GemmParams p{};
            p.X = u; p.ldx = d; p.W = m->ltensor(l, PB_T_W1); p.ldw = d; p.M = N; p.N = F; p.K1 = d;
            p.bias = m->ltensor(l, PB_T_B1);
            p.C = hbuf; p.ldc = F;
            HIP_TRY(pb::launch_gemm(dt, 2, pb::EPI_RELU, p, gws, s));
        }
        {
            Timed t(m, PB_K_GEMM_FC2);
            pb::GemmParams p{};
            p.X = hbuf; p.ldx = F; p.W = m->ltensor(l, PB_T_W2); p.ldw = F; p.M = N; p.N = d; p.K1 = F;
            p.bias = m->ltensor(l, PB_T_B2);
            p.R = x; p.ldr = d;
            // the next layer's LN1 rides on the split-K reduce when the launcher
            // splits; its weights are read here, so wait for that layer first
            if (l + 1 < l1) {
                if (int rc = wait_layer(l + 1)) return rc;
                p.ln_g = m->ltensor(l + 1, PB_T_LN1_G); p.ln_b = m->ltensor(l + 1, PB_T_LN1_B);
                p.ln_out = u; p.ln_eps = c.ln_eps; p.ln_done = &ln1_ready;
                p.shrink = row_shrink_args(l + 1);
            }
            HIP_TRY(pb::launch_gemm(dt, 3, pb::EPI_RESID, p, gws, s));
        }
    }
    if (l1 < L) {  // hand the hidden state to the next stage
        HIP_TRY(hipMemcpyAsync(st->out, x, (size_t)N * d * 4, hipMemcpyDeviceToDevice, s));
        return PB_OK;
    }
    float* zf = (float*)m->at(a.zf);
    {
        Timed t(m, PB_K_LN);
        HIP_TRY(pb::launch_layernorm(dt, x, T, T - 1, m->gtensor(PB_G_LNF_G), m->gtensor(PB_G_LNF_B), zf,
                                     true, B, d, c.ln_eps, s));
    }
    {
        Timed t(m, PB_K_LM_HEAD);
        HIP_TRY(pb::launch_lm_head(dt, zf, B, m->gtensor(PB_G_EMBED), c.vocab, d,
                                   (float*)m->at(a.logits), (float*)m->at(a.pval), (int*)m->at(a.pidx), s));
    }
    {
        Timed t(m, PB_K_ARGMAX);
        HIP_TRY(pb::launch_argmax((const float*)m->at(a.pval), (const int*)m->at(a.pidx), B, c.vocab,
                                  (int32_t*)m->at(a.outtok), s));
    }
    return PB_OK;
}

// True once every weight the forward pass reads is resident: the last load
// (and adapter attach, when adapters are used) has finished on the device.
bool weights_settled(pb_model* m, bool use_lora) {
    if (!m->streamed) return false;
    {
        std::lock_guard<std::mutex> lk(m->mu);
        if (!m->load_done || m->load_rc || !m->globals_ready) return false;
        for (char r : m->ready)
            if (!r) return false;
    }
    if (hipEventQuery(m->ev_load1) != hipSuccess) return false;
    if (use_lora && (!m->lora_recorded || hipEventQuery(m->ev_lora) != hipSuccess)) return false;
    return true;
}

// The forward pass as one graph launch: the launches of a shape are recorded
// the second time the shape is seen (every kernel argument is a function of
// the shape, the adapter targets in use and the fixed arena; the inputs,
// including the position, live in device memory) and replayed from then on.
// Returns 1 when the caller should launch eagerly instead (first sight).
int forward_graph(pb_model* m, int B, int T, bool use_lora, uint32_t lora_union, bool decode) {
    pb_model::Graph* g = nullptr;
    for (auto& e : m->graphs)
        if (e.B == B && e.T == T && e.decode == decode && e.use_lora == use_lora && e.lora_union == lora_union)
            g = &e;
    if (!g) {
        if (m->graphs.size() >= MAX_GRAPHS) {
            auto old = std::min_element(m->graphs.begin(), m->graphs.end(),
                                        [](const pb_model::Graph& a, const pb_model::Graph& b) {
                                            return a.last_use < b.last_use;
                                        });
            if (old->exec) (void)hipGraphExecDestroy(old->exec);
            m->graphs.erase(old);
        }
        m->graphs.push_back({B, T, decode, use_lora, lora_union, nullptr, ++m->graph_clock});
        return 1;
    }
    g->last_use = ++m->graph_clock;
    hipStream_t s = m->compute;
    if (!g->exec) {
        hipGraph_t graph = nullptr;
        HIP_TRY(hipStreamBeginCapture(s, hipStreamCaptureModeRelaxed));
        const int rc = enqueue_forward(m, B, T, use_lora, lora_union, decode, nullptr, false);
        const hipError_t e = hipStreamEndCapture(s, &graph);
        if (rc || e != hipSuccess) {
            if (graph) (void)hipGraphDestroy(graph);
            return rc ? rc : fail(PB_EHIP, "recording the forward pass failed: %s", hipGetErrorString(e));
        }
        hipGraphExec_t exec = nullptr;
        const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
        (void)hipGraphDestroy(graph);
        if (ei != hipSuccess) return fail(PB_EHIP, "hipGraphInstantiate failed: %s", hipGetErrorString(ei));
        g->exec = exec;
    }
    HIP_TRY(hipGraphLaunch(g->exec, s));
    return PB_OK;
}

}  // namespace

// Validate, stage the small inputs, enqueue the forward pass and return the
// greedy tokens (and logits) of B sequences of T new tokens at position pos0.
static int run_forward(pb_model* m, const int32_t* tokens, int32_t B, int32_t T,
                       const int32_t* adapter_of_seq, int32_t* out_tokens, float* out_logits, int pos0,
                       bool decode, const uint8_t* has_kv = nullptr, const Stage* st = nullptr) {
    const pb_config& c = m->cfg;
    const int N = B * T;
    for (int i = 0; i < N; ++i)
        if (tokens[i] < 0 || tokens[i] >= c.vocab) return fail(PB_EINVAL, "token %d at %d outside [0, %d)", tokens[i], i, c.vocab);
    bool use_lora = false;
    uint32_t lora_union = 0;
    for (int b = 0; b < B; ++b) {
        const int a = adapter_of_seq ? adapter_of_seq[b] : -1;
        if (a < -1 || a >= c.max_adapters) return fail(PB_EINVAL, "adapter %d of sequence %d outside [-1, %d)", a, b, c.max_adapters);
        if (a >= 0) {
            if (m->merged_slot >= 0)
                return fail(PB_ESTATE, "adapter %d is merged into the base weights: sequences run with adapter -1",
                            m->merged_slot);
            if (!m->slot_valid[a]) return fail(PB_ESTATE, "adapter slot %d holds no adapter", a);
            use_lora = true;
            lora_union |= m->slot_mask[a];
        }
        for (int t = 0; t < T; ++t) m->h_rowslot[b * T + t] = a;
    }
    std::memcpy(m->h_tokens, tokens, (size_t)N * 4);
    for (int s = 0; s < MAX_SLOTS; ++s) m->h_scale[s] = m->slot_valid[s] ? m->slot_scale[s] : 0.f;
    std::memcpy(&m->h_scale[MAX_SLOTS], &pos0, 4);
    const ArenaLayout& a = m->lay;
    hipStream_t s = m->compute;
    m->tused = 0;
    HIP_TRY(hipMemcpyAsync(m->at(a.tokens), m->h_tokens, (size_t)N * 4, hipMemcpyHostToDevice, s));
    HIP_TRY(hipMemcpyAsync(m->at(a.rowslot), m->h_rowslot, (size_t)N * 4, hipMemcpyHostToDevice, s));
    HIP_TRY(hipMemcpyAsync(m->at(a.slotscale), m->h_scale, SMALL_WORDS * 4, hipMemcpyHostToDevice, s));
    int rc = 1;
    if (m->graphs_on && !m->timing && !has_kv && !st && weights_settled(m, use_lora))
        rc = forward_graph(m, B, T, use_lora, lora_union, decode);
    if (rc == 1) rc = enqueue_forward(m, B, T, use_lora, lora_union, decode, has_kv, true, st);
    if (rc) {
        (void)hipStreamSynchronize(s);
        return rc;
    }
    const bool head = !st || st->l1 == c.n_layers;  // this call ends with the first tokens
    if (head) {
        HIP_TRY(hipMemcpyAsync(m->h_outtok, m->at(a.outtok), (size_t)B * 4, hipMemcpyDeviceToHost, s));
        if (out_logits)
            HIP_TRY(hipMemcpyAsync(m->h_logits, m->at(a.logits), (size_t)B * c.vocab * 4, hipMemcpyDeviceToHost,
                                   s));
    }
    HIP_TRY(hipStreamSynchronize(s));
    if (head) {
        std::memcpy(out_tokens, m->h_outtok, (size_t)B * 4);
        if (out_logits) std::memcpy(out_logits, m->h_logits, (size_t)B * c.vocab * 4);
    }
    if (m->timing) {
        for (size_t i = 0; i + 1 < m->tused; i += 2) {
            float ms = 0.f;
            HIP_TRY(hipEventElapsedTime(&ms, m->tev[i], m->tev[i + 1]));
            const int k = m->tkind[i / 2];
            m->ttotal[k] += ms;
            m->tcount[k] += 1;
        }
    }
    return PB_OK;
}

extern "C" int pb_prefill_first_token(pb_model* m, const int32_t* tokens, int32_t B, int32_t T,
                                      const int32_t* adapter_of_seq, int32_t* out_tokens,
                                      float* out_logits) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    const pb_config& c = m->cfg;
    if (!tokens || !out_tokens) return fail(PB_EINVAL, "tokens and out_tokens must be non-NULL");
    if (B < 1 || B > c.max_batch) return fail(PB_EINVAL, "B=%d outside [1, %d]", B, c.max_batch);
    if (T < 1 || T > c.max_pos) return fail(PB_EINVAL, "T=%d outside [1, %d]", T, c.max_pos);
    if ((int64_t)B * T > c.max_tokens) return fail(PB_EINVAL, "B*T=%lld exceeds max_tokens=%d", (long long)B * T, c.max_tokens);
    if (!m->streamed) return fail(PB_ESTATE, "prefill before pb_stream_layers");
    m->dec_B = 0;  // a failed prefill leaves nothing to decode from
    const int rc = run_forward(m, tokens, B, T, adapter_of_seq, out_tokens, out_logits, 0, false);
    if (rc) return rc;
    if (c.max_new_tokens > 0) {
        m->dec_B = B;
        m->dec_len = T;
        m->dec_steps = 0;
        m->dec_adapter.assign(B, -1);
        for (int b = 0; b < B; ++b) m->dec_adapter[b] = adapter_of_seq ? adapter_of_seq[b] : -1;
    }
    return PB_OK;
}

extern "C" int pb_prefill_stage(pb_model* m, const int32_t* tokens, int32_t B, int32_t T,
                                const int32_t* adapter_of_seq, int32_t layer_begin, int32_t layer_end,
                                const float* hidden_in, float* hidden_out, int32_t* out_tokens, float* out_logits) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    const pb_config& c = m->cfg;
    const int L = c.n_layers;
    if (!tokens) return fail(PB_EINVAL, "tokens must be non-NULL");
    if (B < 1 || B > c.max_batch) return fail(PB_EINVAL, "B=%d outside [1, %d]", B, c.max_batch);
    if (T < 1 || T > c.max_pos) return fail(PB_EINVAL, "T=%d outside [1, %d]", T, c.max_pos);
    if ((int64_t)B * T > c.max_tokens) return fail(PB_EINVAL, "B*T=%lld exceeds max_tokens=%d", (long long)B * T, c.max_tokens);
    if (layer_begin < 0 || layer_end <= layer_begin || layer_end > L)
        return fail(PB_EINVAL, "layers [%d, %d) are not a range of 0..%d", layer_begin, layer_end, L);
    if (layer_begin > 0 && !hidden_in) return fail(PB_EINVAL, "a stage after layer 0 needs hidden_in");
    if (layer_end < L && !hidden_out) return fail(PB_EINVAL, "a stage before the last layer needs hidden_out");
    if (layer_end == L && !out_tokens) return fail(PB_EINVAL, "the last stage needs out_tokens");
    if (!m->streamed) return fail(PB_ESTATE, "prefill before pb_stream_layers");
    m->dec_B = 0;  // a stage leaves nothing to decode from
    const Stage st{layer_begin, layer_end, hidden_in, hidden_out};
    return run_forward(m, tokens, B, T, adapter_of_seq, out_tokens, out_logits, 0, false, nullptr, &st);
}

extern "C" int pb_decode_step(pb_model* m, const int32_t* tokens, int32_t B, const int32_t* adapter_of_seq,
                              int32_t* out_tokens, float* out_logits) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    const pb_config& c = m->cfg;
    if (!tokens || !out_tokens) return fail(PB_EINVAL, "tokens and out_tokens must be non-NULL");
    if (c.max_new_tokens <= 0) return fail(PB_ESTATE, "the model was created without a KV cache (max_new_tokens = 0)");
    if (m->dec_B == 0) return fail(PB_ESTATE, "decode step without a prefill to continue");
    if (B != m->dec_B) return fail(PB_EINVAL, "B=%d differs from the prefill's %d sequences", B, m->dec_B);
    for (int b = 0; b < B; ++b) {
        const int a = adapter_of_seq ? adapter_of_seq[b] : -1;
        if (a != m->dec_adapter[b]) return fail(PB_EINVAL, "sequence %d changed adapter since its prefill", b);
    }
    if (m->dec_steps >= c.max_new_tokens) return fail(PB_ESTATE, "max_new_tokens=%d reached", c.max_new_tokens);
    if (m->dec_len >= c.max_pos) return fail(PB_ESTATE, "sequences already hold max_pos=%d tokens", c.max_pos);
    const int rc = run_forward(m, tokens, B, 1, adapter_of_seq, out_tokens, out_logits, m->dec_len, true);
    if (rc) return rc;
    m->dec_len += 1;
    m->dec_steps += 1;
    return PB_OK;
}

extern "C" int pb_rebuild_kv(pb_model* m, const int32_t* tokens, int32_t B, int32_t T,
                             const int32_t* adapter_of_seq, const uint8_t* layer_has_kv,
                             int32_t* out_tokens, float* out_logits) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    const pb_config& c = m->cfg;
    if (!tokens || !out_tokens || !layer_has_kv) return fail(PB_EINVAL, "NULL argument");
    if (c.max_new_tokens <= 0) return fail(PB_ESTATE, "the model was created without a KV cache (max_new_tokens = 0)");
    if (B < 1 || B > c.max_batch) return fail(PB_EINVAL, "B=%d outside [1, %d]", B, c.max_batch);
    if (T < 1 || T > c.max_pos) return fail(PB_EINVAL, "T=%d outside [1, %d]", T, c.max_pos);
    if ((int64_t)B * T > c.max_tokens) return fail(PB_EINVAL, "B*T=%lld exceeds max_tokens=%d", (long long)B * T, c.max_tokens);
    if (!m->streamed) return fail(PB_ESTATE, "rebuild before pb_stream_layers");
    m->dec_B = 0;
    const int rc = run_forward(m, tokens, B, T, adapter_of_seq, out_tokens, out_logits, 0, false, layer_has_kv);
    if (rc) return rc;
    m->dec_B = B;
    m->dec_len = T;
    m->dec_steps = 0;
    m->dec_adapter.assign(B, -1);
    for (int b = 0; b < B; ++b) m->dec_adapter[b] = adapter_of_seq ? adapter_of_seq[b] : -1;
    return PB_OK;
}

extern "C" int pb_plan_loading(int32_t n_layers, int32_t n_gpus, const uint8_t* alive, int32_t* order,
                               int32_t* block_first, int32_t* block_len) {
    if (n_layers < 1 || n_gpus < 1 || !alive || !order) return fail(PB_EINVAL, "bad arguments");
    std::vector<int> live;
    for (int g = 0; g < n_gpus; ++g)
        if (alive[g]) live.push_back(g);
    if (live.empty()) return fail(PB_EINVAL, "no GPU is alive");
    const int n = (int)live.size();
    for (int g = 0; g < n_gpus; ++g) {
        for (int i = 0; i < n_layers; ++i) order[(size_t)g * n_layers + i] = -1;
        if (block_first) block_first[g] = -1;
        if (block_len) block_len[g] = 0;
    }
    // load balance: block sizes differ by at most one (earlier blocks take the
    // remainder); layer contiguity: block k is one run of layers, in the
    // order of the alive GPUs; each GPU loads its block, then the layers
    // after it, cyclically
    int first = 0;
    for (int k = 0; k < n; ++k) {
        const int len = n_layers / n + (k < n_layers % n ? 1 : 0);
        const int g = live[k];
        for (int i = 0; i < n_layers; ++i) order[(size_t)g * n_layers + i] = (first + i) % n_layers;
        if (block_first) block_first[g] = first;
        if (block_len) block_len[g] = len;
        first += len;
    }
    return PB_OK;
}

// Copy every layer's Wq|Wk|Wv|Wo between the layer blobs and the shadow (one
// strided copy on the compute stream).
static int copy_shadow(pb_model* m, bool to_shadow) {
    const ArenaLayout& a = m->lay;
    char* layers = m->at(a.layers) + a.attn_w;
    char* shadow = m->at(a.shadow);
    if (to_shadow)
        HIP_TRY(hipMemcpy2DAsync(shadow, a.shadow_layer, layers, a.layer_bytes, a.shadow_layer, m->cfg.n_layers,
                                 hipMemcpyDeviceToDevice, m->compute));
    else
        HIP_TRY(hipMemcpy2DAsync(layers, a.layer_bytes, shadow, a.shadow_layer, a.shadow_layer, m->cfg.n_layers,
                                 hipMemcpyDeviceToDevice, m->compute));
    return PB_OK;
}

extern "C" int pb_merge_lora(pb_model* m, int32_t slot) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    const pb_config& c = m->cfg;
    if (slot < 0 || slot >= c.max_adapters) return fail(PB_EINVAL, "slot %d outside [0, %d)", slot, c.max_adapters);
    if (!m->slot_valid[slot]) return fail(PB_ESTATE, "adapter slot %d holds no adapter", slot);
    if (!m->streamed) return fail(PB_ESTATE, "merge before pb_stream_layers");
    if (m->merged_slot >= 0 && !c.merge_shadow)
        return fail(PB_ESTATE, "adapter %d is already merged; stream the base layers again first (or keep a merge shadow)",
                    m->merged_slot);
    const ArenaLayout& a = m->lay;
    hipStream_t s = m->compute;
    // every layer (and the adapter) must have landed before it is rewritten
    if (m->lora_recorded) HIP_TRY(hipStreamWaitEvent(s, m->ev_lora, 0));
    for (int l = 0; l < c.n_layers; ++l) {
        if (int rc = wait_recorded(m, l)) return rc;
        HIP_TRY(hipStreamWaitEvent(s, m->ev_layer[l], 0));
    }
    if (c.merge_shadow) {
        if (m->merged_slot >= 0) {  // switch: back to the unmerged weights first
            if (int rc = copy_shadow(m, false)) return rc;
        } else if (!m->shadow_valid) {
            if (int rc = copy_shadow(m, true)) return rc;
            m->shadow_valid = true;
        }
    }
    m->merged_slot = -1;
    m->dec_B = 0;  // a KV cache from before the merge belongs to another model
    const int tensor_of[4] = {PB_T_WQ, PB_T_WK, PB_T_WV, PB_T_WO};
    for (int l = 0; l < c.n_layers; ++l) {
        for (int t = 0; t < 4; ++t) {
            if (!((m->slot_mask[slot] >> t) & 1u)) continue;
            const char* At = m->at(a.loraA) + (size_t)l * a.loraA_layer + (size_t)t * a.kw * c.d_model * 2;
            const char* Bt = m->at(a.loraB) + (size_t)l * a.loraB_layer + (size_t)t * c.d_model * a.kw * 2;
            HIP_TRY(pb::launch_lora_merge(c.dtype, m->ltensor(l, tensor_of[t]), At, Bt, c.d_model, a.kw, a.rs, slot,
                                          m->slot_scale[slot], s));
        }
    }
    HIP_TRY(hipStreamSynchronize(s));
    m->merged_slot = slot;
    return PB_OK;
}

extern "C" int pb_unmerge_lora(pb_model* m) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    if (!m->cfg.merge_shadow) return fail(PB_ESTATE, "the model keeps no merge shadow");
    if (m->merged_slot < 0) return fail(PB_ESTATE, "no adapter is merged");
    if (int rc = copy_shadow(m, false)) return rc;
    HIP_TRY(hipStreamSynchronize(m->compute));
    m->merged_slot = -1;
    m->dec_B = 0;
    return PB_OK;
}

extern "C" int pb_invalidate_kv(pb_model* m, const uint8_t* layer_lost, int32_t value) {
    if (!m) return fail(PB_EINVAL, "model is NULL");
    if (!layer_lost) return fail(PB_EINVAL, "layer_lost is NULL");
    const ArenaLayout& a = m->lay;
    if (!a.kv_layer) return fail(PB_ESTATE, "the model has no KV cache");
    for (int l = 0; l < m->cfg.n_layers; ++l)
        if (layer_lost[l])
            HIP_TRY(hipMemsetAsync(m->at(a.kv) + (size_t)l * a.kv_layer * 2, value & 0xFF, a.kv_layer * 2,
                                   m->compute));
    HIP_TRY(hipStreamSynchronize(m->compute));
    return PB_OK;
}

// ---- kernel-level entry points (include/pipeboost_ops.h) -------------------

#include "../../include/pipeboost_ops.h"

namespace {

struct OpLora {
    const void* Z = nullptr;
    int32_t ldz = 0, zs = 0;
    const void* W2 = nullptr;
    int32_t K2 = 0, group = 0;
    uint32_t mask = 0;
};

int op_gemm(int32_t dtype, int32_t epi, const void* X, const void* W, const void* bias, void* C, float* R,
            int32_t M, int32_t N, int32_t K, float qscale, int32_t qcols, const pb::GemmWorkspace& ws,
            void* stream, const OpLora& lo = OpLora()) {
    if (dtype != PB_BF16 && dtype != PB_F16) return fail(PB_EINVAL, "bad dtype %d", dtype);
    if (epi < 0 || epi > 2) return fail(PB_EINVAL, "epilogue %d not in 0..2", epi);
    if (M < 0 || N <= 0 || K <= 0 || N % 64 || K % 64)
        return fail(PB_EINVAL, "shape M=%d N=%d K=%d (N and K must be positive multiples of 64)", M, N, K);
    if (!X || !W || !bias || (epi == 2 ? !R : !C)) return fail(PB_EINVAL, "NULL operand");
    pb::GemmParams p{};
    p.X = X; p.ldx = K; p.W = W; p.ldw = K; p.M = M; p.N = N; p.K1 = K;
    p.bias = bias; p.C = C; p.ldc = N; p.R = R; p.ldr = N; p.qscale = qscale; p.qcols = qcols;
    if (lo.K2 > 0) {
        p.X2 = lo.Z; p.ldx2 = lo.ldz; p.x2_group_stride = lo.zs;
        p.W2 = lo.W2; p.ldw2 = lo.K2; p.K2 = lo.K2; p.group = lo.group; p.k2_mask = lo.mask;
    }
    const int role = epi == 0 ? 0 : (epi == 1 ? 2 : 3);
    const int e = epi == 0 ? pb::EPI_QKV : (epi == 1 ? pb::EPI_RELU : pb::EPI_RESID);
    HIP_TRY(pb::launch_gemm(dtype, role, e, p, ws, (hipStream_t)stream));
    return PB_OK;
}

}  // namespace

extern "C" int pb_op_gemm(int32_t dtype, int32_t epi, const void* X, const void* W, const void* bias,
                          void* C, float* R, int32_t M, int32_t N, int32_t K, float qscale,
                          int32_t qcols, void* workspace, size_t workspace_bytes, void* stream) {
    const pb::GemmWorkspace ws{workspace, workspace ? workspace_bytes : 0};
    return op_gemm(dtype, epi, X, W, bias, C, R, M, N, K, qscale, qcols, ws, stream);
}

extern "C" int pb_op_gemm_lora(int32_t dtype, int32_t epi, const void* X, const void* W, const void* bias,
                               void* C, float* R, int32_t M, int32_t N, int32_t K, const void* Z, int32_t ldz,
                               int32_t zs, const void* W2, int32_t K2, int32_t group, uint32_t group_mask,
                               float qscale, int32_t qcols, void* workspace, size_t workspace_bytes,
                               void* stream) {
    if (!Z || !W2 || K2 <= 0 || K2 % 64 || group <= 0 || group % 256 || ldz <= 0 || zs < 0)
        return fail(PB_EINVAL, "pb_op_gemm_lora: bad LoRA operands (K2=%d group=%d ldz=%d zs=%d)", K2, group, ldz, zs);
    if (N > 0 && group > 0 && (size_t)((N - 1) / group) * zs + K2 > (size_t)ldz)
        return fail(PB_EINVAL, "pb_op_gemm_lora: group blocks of Z past its row (ldz=%d)", ldz);
    OpLora lo;
    lo.Z = Z; lo.ldz = ldz; lo.zs = zs; lo.W2 = W2; lo.K2 = K2; lo.group = group; lo.mask = group_mask;
    const pb::GemmWorkspace ws{workspace, workspace ? workspace_bytes : 0};
    return op_gemm(dtype, epi, X, W, bias, C, R, M, N, K, qscale, qcols, ws, stream, lo);
}

// ---- pb_op_gemm without a caller workspace and without allocating ----------
// The split-K partials go to `scratch`, a device array of this file that every
// GPU the library runs on holds (its own copy, at its own address) until the
// process ends.  In host code the name `scratch` is only the host-side stand-in
// of the array: its device address comes from hipGetSymbolAddress, taken once
// per device with that device current, and only that address is ever handed to
// kernels.  Nothing in the array needs to start at zero: every split writes its
// whole partial tile before the reduce reads it.  Calls on one GPU share the
// array, so calls that overlap on that GPU (other streams, other threads) race.

namespace {

constexpr size_t NOALLOC_SCRATCH_BYTES = size_t(64) << 20;
constexpr int NOALLOC_MAX_DEVICES = 64;

__device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
void* g_scratch_dev[NOALLOC_MAX_DEVICES] = {};  // device address of `scratch`, per device

}  // namespace

extern "C" int pb_op_gemm_noalloc(int32_t dtype, int32_t epi, const void* X, const void* W,
                                  const void* bias, void* C, float* R, int32_t M, int32_t N, int32_t K,
                                  float qscale, int32_t qcols, void* stream) {
    if (M < 0 || N <= 0) return fail(PB_EINVAL, "shape M=%d N=%d", M, N);
    if ((size_t)M * (size_t)N * 4 > NOALLOC_SCRATCH_BYTES)
        return fail(PB_EINVAL,
                    "pb_op_gemm_noalloc: M*N*4 = %zu bytes exceeds the %zu-byte scratch (M*N <= %zu); "
                    "use pb_op_gemm with a workspace",
                    (size_t)M * (size_t)N * 4, NOALLOC_SCRATCH_BYTES, NOALLOC_SCRATCH_BYTES / 4);
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= NOALLOC_MAX_DEVICES) return fail(PB_EINVAL, "device %d out of range", dev);
    void* ptr = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_scratch_mu);
        if (!g_scratch_dev[dev]) {
            void* a = nullptr;
            const hipError_t e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
            if (e != hipSuccess || !a)
                return fail(PB_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                            hipGetErrorString(e));
            g_scratch_dev[dev] = a;
        }
        ptr = g_scratch_dev[dev];
    }
    const pb::GemmWorkspace ws{ptr, NOALLOC_SCRATCH_BYTES};
    return op_gemm(dtype, epi, X, W, bias, C, R, M, N, K, qscale, qcols, ws, stream);
}

extern "C" int pb_op_attention(int32_t dtype, const void* qkv, void* out, int32_t B, int32_t T,
                               int32_t H, int32_t hd, void* stream) {
    if (dtype != PB_BF16 && dtype != PB_F16) return fail(PB_EINVAL, "bad dtype %d", dtype);
    if (B < 0 || T < 0 || H <= 0 || (hd != 64 && hd != 128)) return fail(PB_EINVAL, "bad attention shape");
    if (!qkv || !out) return fail(PB_EINVAL, "NULL operand");
    HIP_TRY(pb::launch_attention(dtype, qkv, out, B, T, H, hd, (hipStream_t)stream));
    return PB_OK;
}

extern "C" int pb_op_layernorm(int32_t dtype, const float* x, const void* g, const void* b, void* out,
                               int32_t out_f32, int32_t rows, int32_t d, float eps, void* stream) {
    if (dtype != PB_BF16 && dtype != PB_F16) return fail(PB_EINVAL, "bad dtype %d", dtype);
    if (rows < 0 || d <= 0 || d % 4 || d > 16384 || !(eps > 0.f)) return fail(PB_EINVAL, "bad LayerNorm shape");
    if (!x || !g || !b || !out) return fail(PB_EINVAL, "NULL operand");
    HIP_TRY(pb::launch_layernorm(dtype, x, 1, 0, g, b, out, out_f32 != 0, rows, d, eps, (hipStream_t)stream));
    return PB_OK;
}
