// Stage runtime: memory plan, paged KV allocation, weight streaming through reusable HBM slots,
// residency schedule and the per-layer launch sequence.  Implements include/stage.h.
//
// Memory plan (one stage, one GPU):
//   * every layer is two blocks (Section III-D: a layer splits into its MHA and MLP blocks, each
//     offloadable on its own), each a run of bf16 tensors at 256-byte aligned offsets:
//       MHA block: Wqkv [(Hq + 2 Hkv) d, H] (q rows, then k rows, then v rows) | Wo [H, Hq d] | g1 [H]
//       MLP block: Wg [F, H] | Wu [F, H] | Wd [H, F] | g2 [H]
//     so a loaded layer is described once by fixed offsets (the paper's proxy modules,
//     Section III-C: structure bound once, later loads only refill the bytes);
//   * a resident block owns HBM; an offloaded block owns pinned host memory (hipHostMalloc) and
//     is copied into one of n_stream_slots HBM slots when a call needs it.  A slot holds one
//     layer: its MHA block at offset 0, its MLP block after it;
//   * the KV cache is one pool of 16-token blocks per layer, [block][K|V][Hkv][16][d], shared by
//     all sequences through per-sequence block tables (one table row per sequence, the same block
//     ids in every layer);
//   * RoPE cos/sin tables [max_context][d/2] (fp32, computed in double on the host).
//
// Streaming (Section III-A/III-C): in each call the layers with an offloaded block are loaded
// once, in ascending order; load k of the stage's life goes to slot k mod S.  The copy stream
// waits on the slot's "free" event (recorded by the compute stream after the last kernel that
// read the slot's previous layer), copies the offloaded blocks, MHA first, and records a "ready"
// event per block; the compute stream waits on the MHA block's event before the layer's first
// kernel and on the MLP block's before the MLP kernels, so attention runs while the MLP block
// is still on the link.  With S slots the next S-1 loads proceed while a layer computes, and the
// first loads of a call overlap the call's resident layers.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <memory>
#include <queue>
#include <string>
#include <vector>

#include "stage.h"
#include "stage_kernels.h"

using namespace stg;

namespace stg {
thread_local long long tl_launches = 0;
}

namespace {

constexpr int kDecodeSplitKeys = 64;
constexpr int kMaxContext = 16384;  // decode attention merges at most 256 splits of 64 keys
constexpr int kTimeAll = STAGE_TIME_CALLS | STAGE_TIME_GATEUP | STAGE_TIME_LAYERS;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

constexpr int kMha = 0, kMlp = 1;  // block index: MHA (Wqkv, Wo, g1), MLP (Wg, Wu, Wd, g2)

struct Block {
    bool resident = false;
    void *dev = nullptr;       // HBM copy, exactly when resident
    void *host = nullptr;      // pinned host copy: always when offloaded, kept once made
    void *host_dev = nullptr;  // the pinned copy as kernels address it (zero copy)
};

struct Layer {
    bool loaded = false;
    Block blk[2];
    // any block offloaded: the layer takes a slot load in every staged call
    bool streams() const { return loaded && !(blk[kMha].resident && blk[kMlp].resident); }
};

// Residency codes of the C ABI (STAGE_RES_*), per block.
bool code_keeps(int code, int b) {
    return code == STAGE_RES_RESIDENT || (code == STAGE_RES_MHA_OFFLOADED && b == kMlp) ||
           (code == STAGE_RES_MLP_OFFLOADED && b == kMha);
}

int code_of(const Layer &ly) {
    if (!ly.loaded) return -1;
    const bool a = ly.blk[kMha].resident, m = ly.blk[kMlp].resident;
    if (a && m) return STAGE_RES_RESIDENT;
    if (!a && !m) return STAGE_RES_OFFLOADED;
    return a ? STAGE_RES_MLP_OFFLOADED : STAGE_RES_MHA_OFFLOADED;
}

struct TimeRec {
    int kind, layer;
    hipEvent_t a, b;
};

// An event recorded after one park's copies, shared by the blocks that park freed.
struct ParkEvent {
    hipEvent_t e = nullptr;
    ~ParkEvent() {
        if (e) (void)hipEventDestroy(e);
    }
};

}  // namespace

// What a decode lane owns: its stream and the workspaces and row metadata of its calls.  The call
// in flight swaps its lane's state into the stage's own fields (lane 0's live there), so the
// kernels of a call on lane l use lane l's buffers and stream.
struct LaneState {
    hipStream_t cs = nullptr;
    bool own_cs = false;
    CallMeta *d_meta = nullptr;
    size_t ws_rows = 0, part_rows = 0;
    float *ws_qkv = nullptr, *ws_q = nullptr, *ws_attn = nullptr, *ws_h = nullptr;
    uint16_t *ws_pair = nullptr;
    float *ws_part_o = nullptr, *ws_part_ml = nullptr;
    float *ws_split = nullptr, *ws_split_ss = nullptr;
};

struct stage {
    stage_config cfg{};
    int H = 0, Hq = 0, Hkv = 0, D = 0, F = 0, L = 0;
    int qkv_rows = 0;
    hipStream_t cs = nullptr, xs = nullptr;
    bool own_cs = false, own_xs = false;

    // offsets inside the MHA block (wqkv, wo, g1) and inside the MLP block (wg, wu, wd, g2)
    size_t off_wqkv = 0, off_wo = 0, off_wg = 0, off_wu = 0, off_wd = 0, off_g1 = 0, off_g2 = 0;
    size_t blk_bytes[2] = {0, 0};
    size_t blob_bytes = 0;  // one layer: both blocks
    std::vector<Layer> layers;

    std::vector<void *> slots;
    std::vector<hipEvent_t> slot_ready[2], slot_free;
    long long loads = 0, calls = 0;
    // slot tag check (cfg.slot_check): tags [slot][block] = {layer, load}, and the check record
    int *d_slot_tags = nullptr, *d_slot_rec = nullptr;
    long long slot_checks = 0, slot_checks_run = 0, slot_check_failures = 0;
    std::vector<int> slot_log, demotion_log, residency_log;
    int thresholds_applied = 0;
    std::vector<int> base_code;  // the allocation: residency last set by stage_load_layer

    void *kv_pool = nullptr;
    size_t kv_block_bytes = 0, kv_layer_stride = 0;
    int n_blocks = 0, max_blocks = 0, n_seq_slots = 0;
    int *d_table = nullptr;
    CallMeta *d_meta = nullptr;  // row metadata of the call in flight
    std::vector<std::vector<int>> tables;
    std::vector<int> lengths;
    std::priority_queue<int, std::vector<int>, std::greater<int>> free_blocks;

    float *d_cos = nullptr, *d_sin = nullptr;

    size_t ws_rows = 0;
    float *ws_qkv = nullptr, *ws_q = nullptr, *ws_attn = nullptr, *ws_h = nullptr;
    uint16_t *ws_pair = nullptr;  // interleaved bf16 hi/lo pair of a prefill GEMM operand
    size_t part_rows = 0;
    int max_splits = 0;
    float *ws_part_o = nullptr, *ws_part_ml = nullptr;
    float *ws_split = nullptr, *ws_split_ss = nullptr;  // split matrix-core GEMV partials
    void *ws_dense = nullptr;
    size_t ws_dense_bytes = 0;

    std::vector<TimeRec> recs;
    TimeRec open_rec{0, 0, nullptr, nullptr};  // block-kernel interval being timed
    std::vector<hipEvent_t> ev_pool;

    // KV tails parked between calls (Alg. 2 with pinned host memory as the peer)
    std::vector<int> parked;            // tokens parked per sequence
    std::vector<void *> park_host;      // pinned K then V, [L][n][Hkv][d] each, per sequence
    std::vector<void *> park_host_dev;  // the same buffers as kernels address them
    std::vector<hipEvent_t> ready_ev;   // the sequence's unpark finished (copy stream)
    std::vector<char> ready_pending;
    // per KV block: the event of the park whose copies may still read it, until it is taken again
    std::vector<std::shared_ptr<ParkEvent>> block_park;
    long long bytes_parked = 0, bytes_unparked = 0;

    // decode lanes 1 .. n_lanes-1 (index 0 unused: lane 0's state is the stage's own); per sequence,
    // the stream of the last call that touched it and an event recorded at that call's end
    std::vector<LaneState> lanes;
    std::vector<hipStream_t> seq_stream;
    std::vector<hipEvent_t> seq_ev;

    void *scratch = nullptr;  // this device's scratch array (stage_decode_noalloc)
    long long kernel_launches = 0, last_call_kernels = 0;  // kernels enqueued by prefill/decode calls

    long long tok_prefill = 0, tok_decode = 0, bytes_streamed = 0;
    long long bytes_direct = 0;   // offloaded-block bytes read in place by zero-copy kernels
    std::string err;

    int fail(int code, const char *fmt, ...) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        err = buf;
        return code;
    }
    int fail_hip(hipError_t e, const char *what) {
        return fail(STAGE_EHIP, "%s: %s", what, hipGetErrorString(e));
    }
};

#define HIP_TRY(expr)                                              \
    do {                                                           \
        hipError_t e_ = (expr);                                    \
        if (e_ != hipSuccess) return s->fail_hip(e_, #expr);       \
    } while (0)

namespace {

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) (void)hipSetDevice(dev);
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

bool is_device_ptr(const void *p) {
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return attr.type == hipMemoryTypeDevice;
}

int seq_slot(const stage *s, int mb, int b) { return mb * s->cfg.max_batch + b; }

// A stream on a hardware queue of its own.  HIP spreads ordinary streams over a few hardware queues
// that they share (4 per process by default), in creation order; two streams on one queue run
// their work in one order, so a copy stream's wait for a host-to-HBM copy there holds back every
// compute kernel queued after it, and whether weight streaming overlaps compute would depend on
// how many streams the process made before.  A stream created with a compute-unit mask always gets
// a new queue; the mask here enables every compute unit.
hipError_t create_private_stream(int device, hipStream_t *out) {
    int n_cu = 0;
    hipError_t e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return e;
    if (n_cu < 1) return hipErrorInvalidDevice;
    std::vector<uint32_t> mask((size_t)(n_cu + 31) / 32, 0xffffffffu);
    if (n_cu % 32) mask.back() = (1u << (n_cu % 32)) - 1u;
    return hipExtStreamCreateWithCUMask(out, (uint32_t)mask.size(), mask.data());
}

hipEvent_t pooled_event(stage *s) {
    if (!s->ev_pool.empty()) {
        hipEvent_t e = s->ev_pool.back();
        s->ev_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

int sync_all(stage *s) {
    HIP_TRY(hipStreamSynchronize(s->cs));
    HIP_TRY(hipStreamSynchronize(s->xs));
    for (size_t l = 1; l < s->lanes.size(); ++l) HIP_TRY(hipStreamSynchronize(s->lanes[l].cs));
    return STAGE_OK;
}

// Exchanges the stage's call workspaces (lane 0's, or those swapped in) with o's.
void swap_workspaces(stage *s, LaneState &o) {
    std::swap(s->d_meta, o.d_meta);
    std::swap(s->ws_rows, o.ws_rows);
    std::swap(s->part_rows, o.part_rows);
    std::swap(s->ws_qkv, o.ws_qkv);
    std::swap(s->ws_q, o.ws_q);
    std::swap(s->ws_attn, o.ws_attn);
    std::swap(s->ws_h, o.ws_h);
    std::swap(s->ws_pair, o.ws_pair);
    std::swap(s->ws_part_o, o.ws_part_o);
    std::swap(s->ws_part_ml, o.ws_part_ml);
    std::swap(s->ws_split, o.ws_split);
    std::swap(s->ws_split_ss, o.ws_split_ss);
}

// Exchanges the stage's call state (lane 0's, or the lane swapped in) with lanes[l]'s.
void swap_lane(stage *s, int l) {
    std::swap(s->cs, s->lanes[l].cs);
    swap_workspaces(s, s->lanes[l]);
}

// With several lanes: the call about to run on s->cs waits for the last call on another stream
// that touched any of its sequences (KV cache order); after it, its sequences remember s->cs.
int order_sequences(stage *s, const std::vector<int> &slots) {
    if (s->lanes.size() < 2) return STAGE_OK;
    for (int sl : slots)
        if (s->seq_stream[sl] && s->seq_stream[sl] != s->cs) HIP_TRY(hipStreamWaitEvent(s->cs, s->seq_ev[sl], 0));
    return STAGE_OK;
}
// Entry points that change state outside the call sequence wait for every lane's work first.
int join_lanes(stage *s) { return s->lanes.size() > 1 ? sync_all(s) : STAGE_OK; }

int mark_sequences(stage *s, const std::vector<int> &slots) {
    if (s->lanes.size() < 2) return STAGE_OK;
    for (int sl : slots) {
        HIP_TRY(hipEventRecord(s->seq_ev[sl], s->cs));
        s->seq_stream[sl] = s->cs;
    }
    return STAGE_OK;
}

int ensure_slots(stage *s) {
    if (!s->slots.empty()) return STAGE_OK;
    const int S = s->cfg.n_stream_slots;
    if (S < 1) return s->fail(STAGE_EINVAL, "a layer is offloaded but n_stream_slots is 0");
    if (s->cfg.slot_check && !s->d_slot_tags) {
        // first, so that a stage never holds slots without their tags: every tag starts invalid
        // ({-1, -1}: no layer, no load), the record at zero
        const size_t tag_bytes = sizeof(int) * 4 * (size_t)S;
        if (hipMalloc(&s->d_slot_tags, tag_bytes) != hipSuccess || hipMalloc(&s->d_slot_rec, sizeof(int) * 8) != hipSuccess) {
            (void)hipGetLastError();
            if (s->d_slot_tags) (void)hipFree(s->d_slot_tags);
            s->d_slot_tags = nullptr;
            return s->fail(STAGE_ENOMEM, "cannot allocate the slot tags");
        }
        HIP_TRY(hipMemsetAsync(s->d_slot_tags, 0xFF, tag_bytes, s->cs));
        HIP_TRY(hipMemsetAsync(s->d_slot_rec, 0, sizeof(int) * 8, s->cs));
        HIP_TRY(hipStreamSynchronize(s->cs));
    }
    std::vector<void *> sl(S, nullptr);
    std::vector<hipEvent_t> ra(S, nullptr), rm(S, nullptr), fr(S, nullptr);
    for (int i = 0; i < S; ++i) {
        if (hipMalloc(&sl[i], s->blob_bytes) != hipSuccess ||
            hipEventCreateWithFlags(&ra[i], hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&rm[i], hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&fr[i], hipEventDisableTiming) != hipSuccess) {
            (void)hipGetLastError();
            for (int j = 0; j <= i; ++j) {
                if (sl[j]) (void)hipFree(sl[j]);
                for (hipEvent_t e : {ra[j], rm[j], fr[j]})
                    if (e) (void)hipEventDestroy(e);
            }
            return s->fail(STAGE_ENOMEM, "cannot allocate %d stream slots of %zu bytes", S, s->blob_bytes);
        }
    }
    s->slots = sl;
    s->slot_ready[kMha] = ra;
    s->slot_ready[kMlp] = rm;
    s->slot_free = fr;
    return STAGE_OK;
}

int *slot_tag(const stage *s, int slot, int block) { return s->d_slot_tags + 4 * slot + 2 * block; }

// Slot tag check on the compute stream: block `block` of `slot` should hold `layer` from load
// `load`.  where: 0 / 1 before the MHA / MLP block's first kernel, 2 / 3 after the layer's last.
int check_slot_tag(stage *s, int slot, int block, int layer, long long load, int where) {
    int want = (int)(load & 0x7FFFFFFF);
    if (s->cfg.slot_check == 2 && where == 0) want = (int)((load + 1) & 0x7FFFFFFF);  // self-test
    HIP_TRY(launch_slot_tag_check(slot_tag(s, slot, block), slot, layer, want, where, s->d_slot_rec, s->cs));
    s->slot_checks++;
    return STAGE_OK;
}

// HBM bytes held by resident blocks.
size_t resident_bytes(const stage *s) {
    size_t n = 0;
    for (const Layer &l : s->layers)
        for (int b = 0; b < 2; ++b)
            if (l.loaded && l.blk[b].resident) n += s->blk_bytes[b];
    return n;
}

// The weight budget: n_resident_max whole layers' worth of HBM, spent block by block.
size_t budget_bytes(const stage *s) { return (size_t)s->cfg.n_resident_max * s->blob_bytes; }

void free_block(Block &k) {
    if (k.dev) (void)hipFree(k.dev);
    if (k.host) (void)hipHostFree(k.host);
    k = Block();
}

int alloc_dev(stage *s, int b, void **dev) {
    if (hipMalloc(dev, s->blk_bytes[b]) != hipSuccess) {
        (void)hipGetLastError();
        *dev = nullptr;
        return s->fail(STAGE_ENOMEM, "hipMalloc of a %zu-byte weight block failed", s->blk_bytes[b]);
    }
    return STAGE_OK;
}

// Pinned host memory for block b, with its device address for zero copy.
int alloc_host(stage *s, int b, Block *k) {
    if (hipHostMalloc(&k->host, s->blk_bytes[b], hipHostMallocDefault) != hipSuccess) {
        (void)hipGetLastError();
        k->host = nullptr;
        return s->fail(STAGE_ENOMEM, "hipHostMalloc of a %zu-byte weight block failed", s->blk_bytes[b]);
    }
    if (s->cfg.zero_copy) {
        hipError_t e = hipHostGetDevicePointer(&k->host_dev, k->host, 0);
        if (e != hipSuccess) {
            (void)hipHostFree(k->host);
            k->host = k->host_dev = nullptr;
            return s->fail_hip(e, "hipHostGetDevicePointer");
        }
    }
    return STAGE_OK;
}

// A new home for block b at load time: HBM if resident, else pinned host memory.
int alloc_block(stage *s, int b, bool resident, Block *out) {
    Block k;
    k.resident = resident;
    int rc = resident ? alloc_dev(s, b, &k.dev) : alloc_host(s, b, &k);
    if (rc) return rc;
    *out = k;
    return STAGE_OK;
}

// Checks that moving layer `layer` to residency `code` fits the budget and has slots to stream
// through; changes nothing.
int check_residency(stage *s, int layer, int code) {
    const Layer &ly = s->layers[layer];
    size_t bytes = resident_bytes(s);
    for (int b = 0; b < 2; ++b) {
        if (ly.loaded && ly.blk[b].resident) bytes -= s->blk_bytes[b];
        if (code_keeps(code, b)) bytes += s->blk_bytes[b];
    }
    if (bytes > budget_bytes(s))
        return s->fail(STAGE_ENOMEM, "HBM weight budget of %d layers (%zu bytes) exceeded", s->cfg.n_resident_max,
                       budget_bytes(s));
    if (code != STAGE_RES_RESIDENT && !s->cfg.zero_copy) return ensure_slots(s);
    return STAGE_OK;
}

// Moves the blocks of a loaded layer between HBM and pinned host memory (the planner's offload
// action, Section III-E; block granularity, Section III-D).  Weights never change, so a block's
// pinned host copy, once made, is kept: offloading it again only frees its HBM copy, and only a
// reload moves bytes.  Everything a move needs is allocated before anything moves, so a failed
// allocation leaves the layer as it was.
int set_residency(stage *s, int layer, int code) {
    Layer &ly = s->layers[layer];
    if (code_of(ly) == code) return STAGE_OK;
    int rc = check_residency(s, layer, code);
    if (rc) return rc;
    Block fresh[2];  // new HBM copies (reloads) or first host copies (first offloads)
    bool moves[2];
    auto release = [&]() {
        for (Block &k : fresh) free_block(k);
    };
    for (int b = 0; b < 2; ++b) {
        const Block &k = ly.blk[b];
        moves[b] = code_keeps(code, b) != k.resident;
        if (!moves[b]) continue;
        rc = k.resident ? (k.host ? STAGE_OK : alloc_host(s, b, &fresh[b])) : alloc_dev(s, b, &fresh[b].dev);
        if (rc) {
            release();
            return rc;
        }
    }
    rc = sync_all(s);  // no kernel or copy may still read what is freed below
    if (rc) {
        release();
        return rc;
    }
    for (int b = 0; b < 2; ++b) {
        if (!moves[b]) continue;
        Block &k = ly.blk[b];
        if (k.resident) {
            if (fresh[b].host) {
                // on the compute stream, waited for here: the copies of this file never go through the
                // null stream, which a caller's non-blocking compute stream does not wait for
                hipError_t e = hipMemcpyAsync(fresh[b].host, k.dev, s->blk_bytes[b], hipMemcpyDeviceToHost, s->cs);
                if (e == hipSuccess) e = hipStreamSynchronize(s->cs);
                if (e != hipSuccess) {
                    release();
                    return s->fail_hip(e, "copying a weight block to host memory");
                }
                k.host = fresh[b].host;
                k.host_dev = fresh[b].host_dev;
                fresh[b].host = fresh[b].host_dev = nullptr;
            }
            (void)hipFree(k.dev);
            k.dev = nullptr;
            k.resident = false;
        } else {
            hipError_t e = hipMemcpyAsync(fresh[b].dev, k.host, s->blk_bytes[b], hipMemcpyHostToDevice, s->cs);
            if (e == hipSuccess) e = hipStreamSynchronize(s->cs);
            if (e != hipSuccess) {
                release();
                return s->fail_hip(e, "copying a weight block to HBM");
            }
            k.dev = fresh[b].dev;
            fresh[b].dev = nullptr;
            k.resident = true;
        }
    }
    return STAGE_OK;
}

int ensure_workspace(stage *s, size_t rows, bool split_attention) {
    const size_t need_part = split_attention ? rows : 0;
    if (rows <= s->ws_rows && need_part <= s->part_rows) return STAGE_OK;
    int rc = sync_all(s);
    if (rc) return rc;
    if (rows > s->ws_rows) {
        for (void *p : {(void *)s->ws_qkv, (void *)s->ws_q, (void *)s->ws_attn, (void *)s->ws_h, (void *)s->ws_pair})
            if (p) (void)hipFree(p);
        s->ws_qkv = s->ws_q = s->ws_attn = s->ws_h = nullptr;
        s->ws_pair = nullptr;
        s->ws_rows = 0;
        const size_t qd = (size_t)s->Hq * s->D;
        // ws_qkv holds the prefill QKV rows, the gate and up halves side by side, or the pair of h
        const size_t wide = std::max<size_t>(std::max<size_t>(s->qkv_rows, 2 * (size_t)s->F),
                                             (size_t)pair_ld(s->F) / 2);
        const size_t pair = (size_t)pair_ld(std::max<size_t>(std::max<size_t>(s->H, qd), s->F));
        if (hipMalloc(&s->ws_qkv, rows * wide * sizeof(float)) != hipSuccess ||
            hipMalloc(&s->ws_pair, rows * pair * sizeof(uint16_t)) != hipSuccess ||
            hipMalloc(&s->ws_q, rows * qd * sizeof(float)) != hipSuccess ||
            hipMalloc(&s->ws_attn, rows * qd * sizeof(float)) != hipSuccess ||
            hipMalloc(&s->ws_h, rows * (size_t)s->F * sizeof(float)) != hipSuccess) {
            (void)hipGetLastError();
            return s->fail(STAGE_ENOMEM, "workspace for %zu rows does not fit", rows);
        }
        s->ws_rows = rows;
    }
    if (need_part > s->part_rows) {
        if (s->ws_part_o) (void)hipFree(s->ws_part_o);
        if (s->ws_part_ml) (void)hipFree(s->ws_part_ml);
        s->ws_part_o = s->ws_part_ml = nullptr;
        s->part_rows = 0;
        const size_t n = need_part * s->Hq * (size_t)s->max_splits;
        if (hipMalloc(&s->ws_part_o, n * s->D * sizeof(float)) != hipSuccess ||
            hipMalloc(&s->ws_part_ml, n * 2 * sizeof(float)) != hipSuccess) {
            (void)hipGetLastError();
            return s->fail(STAGE_ENOMEM, "attention partials for %zu rows do not fit", need_part);
        }
        s->part_rows = need_part;
    }
    return STAGE_OK;
}

int ensure_dense(stage *s, size_t bytes) {
    if (bytes <= s->ws_dense_bytes) return STAGE_OK;
    int rc = sync_all(s);
    if (rc) return rc;
    if (s->ws_dense) (void)hipFree(s->ws_dense);
    s->ws_dense = nullptr;
    s->ws_dense_bytes = 0;
    if (hipMalloc(&s->ws_dense, bytes) != hipSuccess) {
        (void)hipGetLastError();
        return s->fail(STAGE_ENOMEM, "staging buffer of %zu bytes does not fit", bytes);
    }
    s->ws_dense_bytes = bytes;
    return STAGE_OK;
}

KvView kv_view(stage *s, int layer) {
    KvView v;
    v.pool = static_cast<char *>(s->kv_pool) + (size_t)layer * s->kv_layer_stride;
    v.block_table = s->d_table;
    v.max_blocks = s->max_blocks;
    v.n_kv_heads = s->Hkv;
    v.head_dim = s->D;
    return v;
}

// Blocks a sequence of current length `len` needs to hold `n` more tokens.
int blocks_needed(const stage *s, int slot, int n) {
    const int len = s->lengths[slot];
    const int have = (int)s->tables[slot].size();
    const int want = (len + n + kBlockTokens - 1) / kBlockTokens;
    return want - have;
}

// Takes blocks (lowest free id first) for the listed sequences in order and mirrors the new
// table entries on the device, on stream `st` (the compute stream unless given).  The caller has
// checked that the pool suffices.
int allocate_blocks(stage *s, const std::vector<int> &slots, int n, hipStream_t st = nullptr) {
    std::vector<int> idx, val;
    for (int slot : slots) {
        const int need = blocks_needed(s, slot, n);
        for (int i = 0; i < need; ++i) {
            const int blk = s->free_blocks.top();
            s->free_blocks.pop();
            // a park that freed this block may still be copying it out: compute waits for it
            // (the copy stream runs the park first anyway)
            if (s->block_park[blk]) {
                if (!st || st == s->cs) HIP_TRY(hipStreamWaitEvent(s->cs, s->block_park[blk]->e, 0));
                s->block_park[blk].reset();
            }
            idx.push_back(slot * s->max_blocks + (int)s->tables[slot].size());
            val.push_back(blk);
            s->tables[slot].push_back(blk);
        }
    }
    if (!idx.empty())
        HIP_TRY(launch_table_write(s->d_table, idx.data(), val.data(), (int)idx.size(), st ? st : s->cs));
    return STAGE_OK;
}

void release_tail_blocks(stage *s, int slot, const std::shared_ptr<ParkEvent> &park = nullptr) {
    const int keep = (s->lengths[slot] + kBlockTokens - 1) / kBlockTokens;
    std::vector<int> &t = s->tables[slot];
    while ((int)t.size() > keep) {
        s->free_blocks.push(t.back());
        if (park) s->block_park[t.back()] = park;
        t.pop_back();
    }
}

// K (or V) bytes of n tokens over all layers, dense [L][n][Hkv][d].
size_t tail_bytes(const stage *s, int n) {
    return (size_t)s->L * n * s->Hkv * s->D * (s->cfg.kv_fp32 ? 4 : 2);
}

KvParkArgs kv_park_args(const stage *s, int slot, int pos0, int n, bool to_pool) {
    KvParkArgs a{};
    a.pool_base = s->kv_pool;
    a.layer_stride = s->kv_layer_stride;
    a.block_table = s->d_table;
    a.max_blocks = s->max_blocks;
    a.n_kv_heads = s->Hkv;
    a.head_dim = s->D;
    a.elem_bytes = s->cfg.kv_fp32 ? 4 : 2;
    a.n_layers = s->L;
    a.slot = slot;
    a.pos0 = pos0;
    a.n = n;
    a.host = s->park_host_dev[slot];
    a.to_pool = to_pool;
    return a;
}

KvCopyArgs kv_copy_args(const stage *s, int slot, int pos0, int n, void *dense, bool to_pool) {
    KvCopyArgs a{};
    a.pool_base = s->kv_pool;
    a.layer_stride = s->kv_layer_stride;
    a.block_table = s->d_table;
    a.max_blocks = s->max_blocks;
    a.n_kv_heads = s->Hkv;
    a.head_dim = s->D;
    a.kv_fp32 = s->cfg.kv_fp32;
    a.n_layers = s->L;
    a.slot = slot;
    a.pos0 = pos0;
    a.n = n;
    a.to_pool = to_pool;
    a.k = dense;
    a.v = static_cast<char *>(dense) + tail_bytes(s, n);
    return a;
}

// Copy stream: the parked tail of `slot` returns into new blocks (taken like a call's); its ready
// event is what the sequence's next compute waits on.  The caller has checked the pool.  Blocks
// in the pool are never still read by the compute stream (calls only free blocks through a park,
// whose copies this stream runs first, or synchronously), so nothing here waits for compute.
int enqueue_unpark(stage *s, int slot) {
    const int n = s->parked[slot];
    int rc = allocate_blocks(s, {slot}, n, s->xs);
    if (rc) return rc;
    HIP_TRY(launch_kv_park(kv_park_args(s, slot, s->lengths[slot], n, true), s->xs));
    if (!s->ready_ev[slot] && hipEventCreateWithFlags(&s->ready_ev[slot], hipEventDisableTiming) != hipSuccess)
        return s->fail(STAGE_EHIP, "hipEventCreate failed");
    HIP_TRY(hipEventRecord(s->ready_ev[slot], s->xs));
    s->ready_pending[slot] = 1;
    s->lengths[slot] += n;
    s->parked[slot] = 0;
    s->bytes_unparked += (long long)(2 * tail_bytes(s, n));
    return STAGE_OK;
}

// Before compute-stream work on the listed sequences: their parked tails come back, and the
// compute stream waits for their copies.  (Blocks the work takes from the pool carry their own
// wait, in allocate_blocks.)
int prepare_sequences(stage *s, const std::vector<int> &slots) {
    for (int sl : slots)
        if (s->parked[sl] > 0) {
            int rc = enqueue_unpark(s, sl);
            if (rc) return rc;
        }
    for (int sl : slots)
        if (s->ready_pending[sl]) {
            HIP_TRY(hipStreamWaitEvent(s->cs, s->ready_ev[sl], 0));
            s->ready_pending[sl] = 0;
        }
    return STAGE_OK;
}

int record_event(stage *s, hipStream_t st, hipEvent_t *out) {
    hipEvent_t e = pooled_event(s);
    if (!e) return s->fail(STAGE_EHIP, "hipEventCreate failed");
    HIP_TRY(hipEventRecord(e, st));
    *out = e;
    return STAGE_OK;
}

// Copies the offloaded blocks of `layer` into `slot` (load number `load` of the stage's life), MHA
// block first, each followed by its ready event; with the slot check, each block's tag is
// invalidated before its copy and set after it.
int enqueue_copy(stage *s, int layer, int slot, long long load) {
    HIP_TRY(hipStreamWaitEvent(s->xs, s->slot_free[slot], 0));
    for (int b = 0; b < 2; ++b) {
        const Block &k = s->layers[layer].blk[b];
        if (k.resident) continue;
        TimeRec rec{b == kMha ? 1 : 4, layer, nullptr, nullptr};
        if (s->cfg.timing & STAGE_TIME_CALLS) {
            int rc = record_event(s, s->xs, &rec.a);
            if (rc) return rc;
        }
        char *dst = static_cast<char *>(s->slots[slot]) + (b == kMha ? 0 : s->blk_bytes[kMha]);
        if (s->cfg.slot_check) HIP_TRY(launch_slot_tag_write(slot_tag(s, slot, b), -1, -1, s->xs));
        HIP_TRY(hipMemcpyAsync(dst, k.host, s->blk_bytes[b], hipMemcpyHostToDevice, s->xs));
        if (s->cfg.slot_check)
            HIP_TRY(launch_slot_tag_write(slot_tag(s, slot, b), layer, (int)(load & 0x7FFFFFFF), s->xs));
        HIP_TRY(hipEventRecord(s->slot_ready[b][slot], s->xs));
        if (s->cfg.timing & STAGE_TIME_CALLS) {
            int rc = record_event(s, s->xs, &rec.b);
            if (rc) return rc;
            s->recs.push_back(rec);
        }
        s->bytes_streamed += (long long)s->blk_bytes[b];
    }
    return STAGE_OK;
}

// Where one layer's kernels find its weights: the MHA and MLP block bases, and the event the
// MLP kernels wait on (the MLP block still arriving in a slot) or null.
struct LayerWeights {
    const uint16_t *mha = nullptr, *mlp = nullptr;
    hipEvent_t mlp_ready = nullptr;
    int slot = -1;          // the stream slot of a layer with an offloaded block, else -1
    long long load = -1;    // its load number (slot tag check)
};

int run_layer_kernels(stage *s, int layer, const LayerWeights &w, int rows, int T, const CallMeta *meta,
                      int grid_splits, const float *x_src, float *x_dst);

// One layer's kernels.  Under STAGE_TIME_LAYERS the MHA-block kernels and the MLP-block kernels
// are bracketed by events separately, so that a wait for the MLP block between them is not
// counted as compute.
int run_layer(stage *s, int layer, const LayerWeights &w, int rows, int T, const CallMeta *meta,
              int grid_splits, const float *x_src, float *x_dst) {
    if (!(s->cfg.timing & STAGE_TIME_LAYERS))
        return run_layer_kernels(s, layer, w, rows, T, meta, grid_splits, x_src, x_dst);
    s->open_rec = TimeRec{3, layer, nullptr, nullptr};
    int rc = record_event(s, s->cs, &s->open_rec.a);
    if (rc) return rc;
    rc = run_layer_kernels(s, layer, w, rows, T, meta, grid_splits, x_src, x_dst);
    if (rc) return rc;
    rc = record_event(s, s->cs, &s->open_rec.b);
    if (rc) return rc;
    s->recs.push_back(s->open_rec);
    return STAGE_OK;
}

// Between a layer's MHA-block and MLP-block kernels: closes the MHA timing record, waits for the
// MLP block if it is still arriving in a slot, opens the MLP timing record.
int mlp_boundary(stage *s, int layer, const LayerWeights &w) {
    const bool timed = s->cfg.timing & STAGE_TIME_LAYERS;
    if (timed) {
        int rc = record_event(s, s->cs, &s->open_rec.b);
        if (rc) return rc;
        s->recs.push_back(s->open_rec);
    }
    if (w.mlp_ready) HIP_TRY(hipStreamWaitEvent(s->cs, w.mlp_ready, 0));
    if (w.mlp_ready && s->cfg.slot_check) {
        int rc = check_slot_tag(s, w.slot, kMlp, layer, w.load, 1);
        if (rc) return rc;
    }
    if (timed) {
        s->open_rec = TimeRec{5, layer, nullptr, nullptr};
        int rc = record_event(s, s->cs, &s->open_rec.a);
        if (rc) return rc;
    }
    return STAGE_OK;
}

// Prefill (T >= 2): projections on the matrix cores with bf16 hi/lo operand pairs.
int run_layer_prefill(stage *s, int layer, const LayerWeights &w, int rows, int T, const CallMeta *meta,
                      const float *x_src, float *x_dst) {
    const uint16_t *base = w.mha;
    const int H = s->H, F = s->F, qd = s->Hq * s->D;
    const float eps = s->cfg.rms_eps;

    HIP_TRY(launch_rmsnorm_split(x_src, base + s->off_g1 / 2, eps, rows, H, s->ws_pair, pair_ld(H), s->cs));
    GemmArgs q{};
    q.a = s->ws_pair; q.lda = pair_ld(H);
    q.w[0] = base + s->off_wqkv / 2;
    q.out = s->ws_qkv; q.ldo = s->qkv_rows;
    q.M = rows; q.N = s->qkv_rows; q.K = H;
    HIP_TRY(launch_gemm(GEMM_STORE, q, 1, s->cs));

    RopeKvArgs r{};
    r.qkv = s->ws_qkv;
    r.q_out = s->ws_q;
    r.cos_t = s->d_cos;
    r.sin_t = s->d_sin;
    r.kv = kv_view(s, layer);
    r.n_q_heads = s->Hq;
    r.kv_fp32 = s->cfg.kv_fp32;
    r.rows = rows;
    r.meta = meta;
    HIP_TRY(launch_rope_kv_store(r, s->cs));

    AttnArgs at{};
    at.q = s->ws_q;
    at.out = s->ws_attn;
    at.kv = kv_view(s, layer);
    at.n_q_heads = s->Hq;
    at.kv_fp32 = s->cfg.kv_fp32;
    at.rows = rows;
    at.split_keys = 0;
    at.n_seqs = rows / T;
    at.rows_per_seq = T;
    at.meta = meta;
    if (!s->cfg.kv_fp32) {   // the matrix-core kernel writes the O projection's operand pair itself
        at.out_pair = s->ws_pair;
        at.out_pair_ld = pair_ld(qd);
    }
    HIP_TRY(launch_attention(at, s->cs));
    if (s->cfg.kv_fp32) HIP_TRY(launch_split(s->ws_attn, rows, qd, s->ws_pair, pair_ld(qd), s->cs));

    GemmArgs o{};
    o.a = s->ws_pair; o.lda = pair_ld(qd);
    o.w[0] = base + s->off_wo / 2;
    o.out = x_dst; o.res = x_src; o.ldo = H;
    o.M = rows; o.N = H; o.K = qd;
    HIP_TRY(launch_gemm(GEMM_RESIDUAL, o, 1, s->cs));

    base = w.mlp;
    int rc = mlp_boundary(s, layer, w);
    if (rc) return rc;
    HIP_TRY(launch_rmsnorm_split(x_dst, base + s->off_g2 / 2, eps, rows, H, s->ws_pair, pair_ld(H), s->cs));
    GemmArgs gu{};
    gu.a = s->ws_pair; gu.lda = pair_ld(H);
    gu.w[0] = base + s->off_wg / 2;
    gu.w[1] = base + s->off_wu / 2;
    gu.M = rows; gu.N = F; gu.K = H;
    const uint16_t *h = s->ws_pair;   // h = silu(Wg y) * (Wu y) as a bf16 pair
    if (H % 32 == 0) {
        // SwiGLU and the hi/lo split in the GEMM's epilogue; the GEMM still reads the pair of y
        // from ws_pair, so h goes to the (fp32-sized) QKV workspace
        gu.out_pair = reinterpret_cast<uint16_t *>(s->ws_qkv);
        gu.ldo = pair_ld(F);
        HIP_TRY(launch_gemm(GEMM_SWIGLU, gu, 1, s->cs));
        h = gu.out_pair;
    } else {
        gu.out = s->ws_qkv; gu.ldo = 2 * (long)F;
        gu.out_col[0] = 0; gu.out_col[1] = F;
        HIP_TRY(launch_gemm(GEMM_STORE, gu, 2, s->cs));
        HIP_TRY(launch_swiglu_split(s->ws_qkv, F, rows, s->ws_pair, pair_ld(F), s->cs));
    }

    GemmArgs dn{};
    dn.a = h; dn.lda = pair_ld(F);
    dn.w[0] = base + s->off_wd / 2;
    dn.out = x_dst; dn.res = x_dst; dn.ldo = H;
    dn.M = rows; dn.N = H; dn.K = F;
    HIP_TRY(launch_gemm(GEMM_RESIDUAL, dn, 1, s->cs));
    return STAGE_OK;
}

int run_layer_kernels(stage *s, int layer, const LayerWeights &w, int rows, int T, const CallMeta *meta,
                      int grid_splits, const float *x_src, float *x_dst) {
    if (T >= 2) return run_layer_prefill(s, layer, w, rows, T, meta, x_src, x_dst);
    if ((size_t)rows > s->part_rows || !s->ws_part_o || !s->ws_part_ml)
        return s->fail(STAGE_ESTATE, "attention partials sized for %zu rows, call has %d", s->part_rows, rows);
    const uint16_t *base = w.mha, *mlp = w.mlp;
    const size_t qd = (size_t)s->Hq * s->D;

    GemvArgs q{};
    q.w = base + s->off_wqkv / 2;
    q.act = x_src;
    q.act_ld = s->H;
    q.gain = base + s->off_g1 / 2;
    q.out = s->ws_q;
    q.out_ld = (long)qd;
    q.N = s->qkv_rows;
    q.K = s->H;
    q.rows = rows;
    q.eps = s->cfg.rms_eps;
    q.cos_t = s->d_cos;
    q.sin_t = s->d_sin;
    q.kv = kv_view(s, layer);
    q.n_q_heads = s->Hq;
    q.kv_fp32 = s->cfg.kv_fp32;
    q.meta = meta;
    q.split_part = s->ws_split;  // matrix-core launches may split K
    q.split_ss = s->ws_split_ss;

    AttnArgs at{};
    at.q = s->ws_q;
    at.out = s->ws_attn;
    at.part_o = s->ws_part_o;
    at.part_ml = s->ws_part_ml;
    at.kv = kv_view(s, layer);
    at.n_q_heads = s->Hq;
    at.kv_fp32 = s->cfg.kv_fp32;
    at.rows = rows;
    at.split_keys = kDecodeSplitKeys;
    at.max_splits = s->max_splits;
    at.grid_splits = grid_splits;
    at.n_seqs = rows;        // decode: one row per sequence
    at.rows_per_seq = 1;
    at.meta = meta;

    GemvArgs o{};
    o.w = base + s->off_wo / 2;
    o.act = s->ws_attn;
    o.act_ld = (long)qd;
    o.res = x_src;
    o.out = x_dst;
    o.out_ld = s->H;
    o.N = s->H;
    o.K = (int)qd;
    o.rows = rows;
    o.split_part = s->ws_split;
    o.split_ss = s->ws_split_ss;

    GemvArgs gu{};
    gu.w = mlp + s->off_wg / 2;
    gu.w2 = mlp + s->off_wu / 2;
    gu.act = x_dst;
    gu.act_ld = s->H;
    gu.gain = mlp + s->off_g2 / 2;
    gu.out = s->ws_h;
    gu.out_ld = s->F;
    gu.N = s->F;
    gu.K = s->H;
    gu.rows = rows;
    gu.eps = s->cfg.rms_eps;
    gu.split_part = s->ws_split;
    gu.split_ss = s->ws_split_ss;

    GemvArgs dn{};
    dn.w = mlp + s->off_wd / 2;
    dn.act = s->ws_h;
    dn.act_ld = s->F;
    dn.res = x_dst;
    dn.out = x_dst;
    dn.out_ld = s->H;
    dn.N = s->H;
    dn.K = s->F;
    dn.rows = rows;
    dn.split_part = s->ws_split;
    dn.split_ss = s->ws_split_ss;

    // Timed kernel: the gate/up projection of one layer per call (rotating), so that the events
    // barely perturb the step.
    TimeRec rec{2, layer, nullptr, nullptr};
    if ((s->cfg.timing & STAGE_TIME_GATEUP) && layer == (int)((s->calls - 1) % s->L)) {
        rec.a = pooled_event(s);
        rec.b = pooled_event(s);
        if (!rec.a || !rec.b) return s->fail(STAGE_EHIP, "hipEventCreate failed");
    }
    HIP_TRY(launch_gemv(GEMV_NORM_ROPE_KV, q, s->cs));
    HIP_TRY(launch_attention(at, s->cs));
    HIP_TRY(launch_gemv(GEMV_PLAIN_RESIDUAL, o, s->cs));
    int rc = mlp_boundary(s, layer, w);
    if (rc) return rc;
    HIP_TRY(launch_gemv(GEMV_NORM_SWIGLU, gu, s->cs, rec.a, rec.b));
    HIP_TRY(launch_gemv(GEMV_PLAIN_RESIDUAL, dn, s->cs));
    if (rec.a) s->recs.push_back(rec);
    return STAGE_OK;
}

// Planner steps (plan_mode 1): the step that holds `held` tokens offloads alpha MHA and beta MLP
// blocks beyond the allocation, the highest-id layers first (Section III-E, Eq. (7)); layers whose
// residency differs from that target move, ascending.  The target keeps a subset of the
// allocation's resident blocks, so it always fits the budget the allocation fits.
std::vector<int> plan_codes(const stage *s, long long held) {
    const stage_config &c = s->cfg;
    int step = -1;
    for (int j = 0; j < c.n_thresholds; ++j)
        if (c.thresholds[j] <= held) step = j;
    int alpha = step < 0 ? 0 : c.plan_alpha[step], beta = step < 0 ? 0 : c.plan_beta[step];
    std::vector<bool> keep_a(s->L), keep_m(s->L);
    for (int l = 0; l < s->L; ++l) {
        keep_a[l] = code_keeps(s->base_code[l], kMha);
        keep_m[l] = code_keeps(s->base_code[l], kMlp);
    }
    for (int l = s->L - 1; l >= 0 && alpha > 0; --l)
        if (keep_a[l]) { keep_a[l] = false; --alpha; }
    for (int l = s->L - 1; l >= 0 && beta > 0; --l)
        if (keep_m[l]) { keep_m[l] = false; --beta; }
    std::vector<int> codes(s->L);
    for (int l = 0; l < s->L; ++l)
        codes[l] = keep_a[l] ? (keep_m[l] ? STAGE_RES_RESIDENT : STAGE_RES_MLP_OFFLOADED)
                             : (keep_m[l] ? STAGE_RES_MHA_OFFLOADED : STAGE_RES_OFFLOADED);
    return codes;
}

int apply_plan(stage *s, long long call_no, long long held) {
    const std::vector<int> codes = plan_codes(s, held);
    for (int l = 0; l < s->L; ++l) {
        const int code = codes[l];
        if (code == code_of(s->layers[l])) continue;
        int rc = set_residency(s, l, code);
        if (rc) return rc;
        for (int v : {(int)call_no, l, code}) s->residency_log.push_back(v);
    }
    return STAGE_OK;
}

int run_call_body(stage *s, int n_mb, const int32_t *mb_ids, int B, int T, const float *x_in, float *x_out,
                  bool decode);

// Shared body of prefill and decode; counts the kernels the call enqueues.
int run_call(stage *s, int n_mb, const int32_t *mb_ids, int B, int T, const float *x_in, float *x_out,
             bool decode) {
    const long long before = tl_launches;
    const int rc = run_call_body(s, n_mb, mb_ids, B, T, x_in, x_out, decode);
    if (s) {
        s->last_call_kernels = tl_launches - before;
        s->kernel_launches += s->last_call_kernels;
    }
    return rc;
}

int run_call_body(stage *s, int n_mb, const int32_t *mb_ids, int B, int T, const float *x_in, float *x_out,
                  bool decode) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    const stage_config &c = s->cfg;
    if (n_mb < 1 || n_mb > c.max_microbatches || !mb_ids || B < 1 || B > c.max_batch || T < 1 ||
        !x_in || !x_out)
        return s->fail(STAGE_EINVAL, "bad call arguments (n_mb=%d B=%d T=%d)", n_mb, B, T);
    std::vector<int> slots;
    std::vector<char> seen(c.max_microbatches, 0);
    for (int k = 0; k < n_mb; ++k) {
        const int mb = mb_ids[k];
        if (mb < 0 || mb >= c.max_microbatches || seen[mb])
            return s->fail(STAGE_EINVAL, "micro-batch id %d out of range or repeated", mb);
        seen[mb] = 1;
        for (int b = 0; b < B; ++b) slots.push_back(seq_slot(s, mb, b));
    }
    for (int l = 0; l < s->L; ++l)
        if (!s->layers[l].loaded) return s->fail(STAGE_EINVAL, "layer %d is not loaded", l);
    int longest = 0;
    for (int len : s->lengths) longest = std::max(longest, len);
    int need_blocks = 0;
    for (int sl : slots) {
        const int len = s->lengths[sl] + s->parked[sl];  // a parked tail comes back first
        if (decode && len < 1)
            return s->fail(STAGE_ESTATE, "decode on an empty sequence (slot %d)", sl);
        if (len + T > c.max_context)
            return s->fail(STAGE_ERANGE, "sequence would exceed max_context %d", c.max_context);
        need_blocks += blocks_needed(s, sl, s->parked[sl] + T);
        longest = std::max(longest, len + T);
    }
    if (need_blocks > (int)s->free_blocks.size())
        return s->fail(STAGE_ENOMEM, "KV pool exhausted (%d blocks needed, %d free)", need_blocks,
                       (int)s->free_blocks.size());
    const size_t rows = (size_t)slots.size() * T;
    DeviceGuard dg(c.device);
    // one row per sequence (a decode, or a one-token prefill) runs the decode kernels, whose
    // attention needs the split partials
    int rc = ensure_workspace(s, rows, T == 1);
    if (rc) return rc;
    // A zero-copy call with one token per sequence runs offloaded layers on their host blobs and
    // stages nothing; in zero-copy mode the slots are allocated by the first call that stages.
    const bool direct = c.zero_copy && T == 1;
    if (!direct && s->slots.empty()) {
        bool may_stream = c.plan_mode ? c.n_thresholds > 0 : s->thresholds_applied < c.n_thresholds;
        for (const Layer &ly : s->layers) may_stream = may_stream || ly.streams();
        if (may_stream) {
            rc = ensure_slots(s);
            if (rc) return rc;
        }
    }

    rc = order_sequences(s, slots);
    if (rc) return rc;
    rc = prepare_sequences(s, slots);
    if (rc) return rc;

    const long long call_no = s->calls;
    if (c.plan_mode) {
        long long held = (long long)rows;
        for (int len : s->lengths) held += len;
        rc = apply_plan(s, call_no, held);
        if (rc) return rc;
    }
    // threshold schedule: thresholds reached by this call demote resident layers, highest first
    while (!c.plan_mode && s->thresholds_applied < c.n_thresholds &&
           c.thresholds[s->thresholds_applied] <= longest) {
        s->thresholds_applied++;
        int victim = -1;
        for (int l = s->L - 1; l >= 0; --l)
            if (s->layers[l].blk[kMha].resident || s->layers[l].blk[kMlp].resident) { victim = l; break; }
        if (victim < 0) continue;
        rc = set_residency(s, victim, STAGE_RES_OFFLOADED);
        if (rc) return rc;
        s->demotion_log.push_back((int)call_no);
        s->demotion_log.push_back(victim);
        for (int v : {(int)call_no, victim, (int)STAGE_RES_OFFLOADED}) s->residency_log.push_back(v);
    }

    rc = allocate_blocks(s, slots, T);
    if (rc) return rc;
    CallMeta meta{};
    meta.n_seqs = (int)slots.size();
    meta.rows_per_seq = T;
    int max_ctx = 0;
    for (size_t i = 0; i < slots.size(); ++i) {
        meta.seq_slot[i] = slots[i];
        meta.pos0[i] = s->lengths[slots[i]];
        s->lengths[slots[i]] += T;
        max_ctx = std::max(max_ctx, s->lengths[slots[i]]);
    }
    const int grid_splits = (max_ctx + kDecodeSplitKeys - 1) / kDecodeSplitKeys;
    if (T == 1 && grid_splits > s->max_splits)
        return s->fail(STAGE_ESTATE, "attention partials hold %d splits, the call needs %d", s->max_splits, grid_splits);
    HIP_TRY(launch_meta_write(meta, s->d_meta, s->cs));
    s->calls++;
    if (decode) s->tok_decode += (long long)rows; else s->tok_prefill += (long long)rows;

    TimeRec call_rec{0, -1, nullptr, nullptr};
    if (c.timing & STAGE_TIME_CALLS) {
        rc = record_event(s, s->cs, &call_rec.a);
        if (rc) return rc;
    }

    // streamed layers of this call, ascending; load j -> slot (loads + j) mod S
    std::vector<int> streamed;
    for (int l = 0; l < s->L; ++l)
        if (s->layers[l].streams() && !direct) streamed.push_back(l);
    const int S = c.n_stream_slots;
    const long long load0 = s->loads;
    auto slot_of = [&](int j) { return (int)((load0 + j) % S); };
    const int n_str = (int)streamed.size();
    for (int j = 0; j < n_str; ++j) {
        s->slot_log.push_back((int)call_no);
        s->slot_log.push_back(streamed[j]);
        s->slot_log.push_back(slot_of(j));
    }
    s->loads += n_str;
    for (int j = 0; j < std::min(S, n_str); ++j) {
        rc = enqueue_copy(s, streamed[j], slot_of(j), load0 + j);
        if (rc) return rc;
    }

    int j = 0;
    for (int l = 0; l < s->L; ++l) {
        const float *src = (l == 0) ? x_in : x_out;
        const Layer &ly = s->layers[l];
        LayerWeights w;
        const uint16_t **base[2] = {&w.mha, &w.mlp};
        if (!ly.streams() || direct) {
            for (int b = 0; b < 2; ++b) {
                const Block &k = ly.blk[b];
                if (!k.resident) s->bytes_direct += (long long)s->blk_bytes[b];
                *base[b] = static_cast<const uint16_t *>(k.resident ? k.dev : k.host_dev);
            }
            rc = run_layer(s, l, w, (int)rows, T, s->d_meta, grid_splits, src, x_out);
            if (rc) return rc;
            continue;
        }
        const int sl = slot_of(j);
        const char *slot = static_cast<const char *>(s->slots[sl]);
        for (int b = 0; b < 2; ++b) {
            const Block &k = ly.blk[b];
            *base[b] = reinterpret_cast<const uint16_t *>(
                k.resident ? static_cast<const char *>(k.dev) : slot + (b == kMha ? 0 : s->blk_bytes[kMha]));
        }
        w.slot = sl;
        w.load = load0 + j;
        const bool check = s->cfg.slot_check != 0;
        if (!ly.blk[kMha].resident) {
            HIP_TRY(hipStreamWaitEvent(s->cs, s->slot_ready[kMha][sl], 0));
            if (check && (rc = check_slot_tag(s, sl, kMha, l, w.load, 0))) return rc;
        }
        if (!ly.blk[kMlp].resident) w.mlp_ready = s->slot_ready[kMlp][sl];
        rc = run_layer(s, l, w, (int)rows, T, s->d_meta, grid_splits, src, x_out);
        if (rc) return rc;
        // the layer's kernels are enqueued: its blocks must still hold it (no refill has begun)
        for (int b = 0; b < 2 && check; ++b)
            if (!ly.blk[b].resident && (rc = check_slot_tag(s, sl, b, l, w.load, 2 + b))) return rc;
        HIP_TRY(hipEventRecord(s->slot_free[sl], s->cs));
        if (j + S < n_str) {
            rc = enqueue_copy(s, streamed[j + S], slot_of(j + S), load0 + j + S);
            if (rc) return rc;
        }
        ++j;
    }
    if (c.timing & STAGE_TIME_CALLS) {
        rc = record_event(s, s->cs, &call_rec.b);
        if (rc) return rc;
        s->recs.push_back(call_rec);
    }
    return mark_sequences(s, slots);
}

// Where stage_decode_noalloc puts a call's workspaces in the scratch array: byte offsets, 256-byte
// aligned; `split` and `split_ss` only for calls of 3 rows or more (the matrix-core projections).
struct ScratchLayout {
    size_t meta = 0, q = 0, attn = 0, h = 0, part_o = 0, part_ml = 0, split = 0, split_ss = 0, total = 0;
    bool has_split = false;
};

ScratchLayout scratch_layout(const stage *s, size_t rows, int splits) {
    ScratchLayout p;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = align256(off + bytes);
        return at;
    };
    const size_t qd = (size_t)s->Hq * s->D;
    p.meta = take(sizeof(CallMeta));
    p.q = take(rows * qd * sizeof(float));
    p.attn = take(rows * qd * sizeof(float));
    p.h = take(rows * (size_t)s->F * sizeof(float));
    p.part_o = take(rows * s->Hq * (size_t)splits * s->D * sizeof(float));
    p.part_ml = take(rows * s->Hq * (size_t)splits * 2 * sizeof(float));
    p.has_split = rows >= 3;
    if (p.has_split) {
        const size_t units = std::max<size_t>(std::max<size_t>(s->qkv_rows / 2, s->H), s->F);
        p.split = take(sizeof(float) * kGemvMaxSplits * 2 * 16 * units);
        p.split_ss = take(sizeof(float) * kGemvMaxSplits * 16);
    }
    p.total = off;
    return p;
}
}  // namespace

extern "C" {

void stage_config_default(stage_config *cfg) {
    if (!cfg) return;
    std::memset(cfg, 0, sizeof *cfg);
    cfg->rope_theta = 10000.f;
    cfg->rms_eps = 1e-5f;
    cfg->kv_block_tokens = kBlockTokens;
    cfg->n_stream_slots = 2;
}

const char *stage_strerror(int32_t status) {
    switch (status) {
        case STAGE_OK: return "ok";
        case STAGE_EINVAL: return "invalid argument";
        case STAGE_ENOMEM: return "out of memory (HBM budget, allocation or KV pool)";
        case STAGE_EHIP: return "HIP runtime error";
        case STAGE_ESTATE: return "invalid state for this call";
        case STAGE_ERANGE: return "sequence would exceed max_context";
        case STAGE_ESLOT: return "slot tag check failed";
        default: return "unknown status";
    }
}

const char *stage_last_error(stage *s) { return s ? s->err.c_str() : "null stage handle"; }

int stage_init(const stage_config *cfg, stage **out) {
    if (!cfg || !out) return STAGE_EINVAL;
    *out = nullptr;
    const stage_config &c = *cfg;
    const bool shape_ok = c.n_layers >= 1 && c.hidden >= 8 && c.hidden % 8 == 0 && c.n_q_heads >= 1 &&
                          c.n_kv_heads >= 1 && c.n_q_heads % c.n_kv_heads == 0 && c.head_dim >= 8 &&
                          c.head_dim % 8 == 0 && c.head_dim <= 256 && c.ffn >= 8 && c.ffn % 8 == 0 &&
                          attention_supported(c.n_q_heads / c.n_kv_heads, c.head_dim) &&
                          c.rope_theta > 0.f && c.rms_eps >= 0.f;
    const bool cap_ok = c.max_microbatches >= 1 && c.max_batch >= 1 &&
                        (long)c.max_microbatches * c.max_batch <= kMaxSeqs && c.max_context >= 1 &&
                        c.max_context <= kMaxContext &&
                        c.kv_block_tokens == kBlockTokens && c.kv_pool_blocks >= 0 &&
                        (c.kv_fp32 == 0 || c.kv_fp32 == 1) && c.n_resident_max >= 0 &&
                        c.n_resident_max <= c.n_layers && c.n_stream_slots >= 0 && c.n_stream_slots <= 64 &&
                        c.n_thresholds >= 0 && c.n_thresholds <= STAGE_MAX_THRESHOLDS &&
                        (c.timing & ~kTimeAll) == 0 && (c.zero_copy == 0 || c.zero_copy == 1) &&
                        c.kv_park_tokens >= 0 && c.kv_park_tokens <= c.max_context && c.n_lanes >= 0 &&
                        c.n_lanes <= STAGE_MAX_LANES && c.slot_check >= 0 && c.slot_check <= 2;
    if (!shape_ok || !cap_ok) return STAGE_EINVAL;
    if (c.plan_mode != 0 && c.plan_mode != 1) return STAGE_EINVAL;
    for (int i = 0; i < c.n_thresholds; ++i) {
        if (c.thresholds[i] < (c.plan_mode ? 0 : 1) || (i > 0 && c.thresholds[i] < c.thresholds[i - 1]))
            return STAGE_EINVAL;
        if (c.plan_mode && (c.plan_alpha[i] < 0 || c.plan_beta[i] < 0)) return STAGE_EINVAL;
    }
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || c.device < 0 || c.device >= ndev) {
        (void)hipGetLastError();
        return STAGE_EINVAL;
    }
    DeviceGuard dg(c.device);

    stage *s = new stage();
    s->cfg = c;
    s->L = c.n_layers; s->H = c.hidden; s->Hq = c.n_q_heads; s->Hkv = c.n_kv_heads;
    s->D = c.head_dim; s->F = c.ffn;
    s->qkv_rows = (s->Hq + 2 * s->Hkv) * s->D;
    const size_t H = s->H, F = s->F, qd = (size_t)s->Hq * s->D;
    size_t off = 0;  // MHA block
    s->off_wqkv = off; off = align256(off + (size_t)s->qkv_rows * H * 2);
    s->off_wo = off;   off = align256(off + H * qd * 2);
    s->off_g1 = off;   off = align256(off + H * 2);
    s->blk_bytes[kMha] = off;
    off = 0;         // MLP block
    s->off_wg = off;   off = align256(off + F * H * 2);
    s->off_wu = off;   off = align256(off + F * H * 2);
    s->off_wd = off;   off = align256(off + H * F * 2);
    s->off_g2 = off;   off = align256(off + H * 2);
    s->blk_bytes[kMlp] = off;
    s->blob_bytes = s->blk_bytes[kMha] + s->blk_bytes[kMlp];
    s->layers.assign(s->L, Layer());
    s->base_code.assign(s->L, STAGE_RES_OFFLOADED);

    s->n_seq_slots = c.max_microbatches * c.max_batch;
    s->max_blocks = (c.max_context + kBlockTokens - 1) / kBlockTokens;
    s->n_blocks = c.kv_pool_blocks > 0 ? c.kv_pool_blocks : s->n_seq_slots * s->max_blocks;
    s->kv_block_bytes = (size_t)2 * s->Hkv * kBlockTokens * s->D * (c.kv_fp32 ? 4 : 2);
    s->kv_layer_stride = align256(s->kv_block_bytes * s->n_blocks);
    s->max_splits = (c.max_context + kDecodeSplitKeys - 1) / kDecodeSplitKeys;
    s->tables.assign(s->n_seq_slots, {});
    s->lengths.assign(s->n_seq_slots, 0);
    s->parked.assign(s->n_seq_slots, 0);
    s->park_host.assign(s->n_seq_slots, nullptr);
    s->park_host_dev.assign(s->n_seq_slots, nullptr);
    s->ready_ev.assign(s->n_seq_slots, nullptr);
    s->ready_pending.assign(s->n_seq_slots, 0);
    for (int b = 0; b < s->n_blocks; ++b) s->free_blocks.push(b);

    auto cleanup = [&](int code) {
        stage_destroy(s);
        return code;
    };
    if (c.compute_stream) s->cs = static_cast<hipStream_t>(c.compute_stream);
    else if (create_private_stream(c.device, &s->cs) == hipSuccess) s->own_cs = true;
    else return cleanup(STAGE_EHIP);
    if (c.copy_stream) s->xs = static_cast<hipStream_t>(c.copy_stream);
    else if (create_private_stream(c.device, &s->xs) == hipSuccess) s->own_xs = true;
    else return cleanup(STAGE_EHIP);

    if (scratch_setup(c.device, &s->scratch) != hipSuccess) return cleanup(STAGE_EHIP);
    if (hipMalloc(&s->kv_pool, s->kv_layer_stride * s->L) != hipSuccess ||
        hipMalloc(&s->d_table, sizeof(int) * (size_t)s->n_seq_slots * s->max_blocks) != hipSuccess ||
        hipMalloc(&s->d_cos, sizeof(float) * (size_t)c.max_context * (s->D / 2)) != hipSuccess ||
        hipMalloc(&s->d_sin, sizeof(float) * (size_t)c.max_context * (s->D / 2)) != hipSuccess ||
        hipMalloc(&s->d_meta, sizeof(CallMeta)) != hipSuccess ||
        hipMalloc(&s->ws_split, sizeof(float) * kGemvMaxSplits * 2 * 16 *
                                    std::max<size_t>(std::max<size_t>(s->qkv_rows / 2, s->H), s->F)) != hipSuccess ||
        hipMalloc(&s->ws_split_ss, sizeof(float) * kGemvMaxSplits * 16) != hipSuccess) {
        (void)hipGetLastError();
        return cleanup(STAGE_ENOMEM);
    }
    s->block_park.assign(s->n_blocks, nullptr);
    if (hipMemsetAsync(s->d_table, 0, sizeof(int) * (size_t)s->n_seq_slots * s->max_blocks, s->cs) != hipSuccess)
        return cleanup(STAGE_EHIP);
    if (c.n_lanes > 1) {
        s->lanes.resize(c.n_lanes);
        for (int l = 1; l < c.n_lanes; ++l) {
            LaneState &ln = s->lanes[l];
            if (c.lane_streams[l]) ln.cs = static_cast<hipStream_t>(c.lane_streams[l]);
            else if (create_private_stream(c.device, &ln.cs) == hipSuccess) ln.own_cs = true;
            else return cleanup(STAGE_EHIP);
            if (hipMalloc(&ln.d_meta, sizeof(CallMeta)) != hipSuccess ||
                hipMalloc(&ln.ws_split, sizeof(float) * kGemvMaxSplits * 2 * 16 *
                                            std::max<size_t>(std::max<size_t>(s->qkv_rows / 2, s->H), s->F)) != hipSuccess ||
                hipMalloc(&ln.ws_split_ss, sizeof(float) * kGemvMaxSplits * 16) != hipSuccess) {
                (void)hipGetLastError();
                return cleanup(STAGE_ENOMEM);
            }
        }
        s->seq_stream.assign(s->n_seq_slots, nullptr);
        s->seq_ev.assign(s->n_seq_slots, nullptr);
        for (hipEvent_t &e : s->seq_ev)
            if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return cleanup(STAGE_EHIP);
    }
    // RoPE tables: angle = p * theta^(-2i/d), evaluated in double, cos/sin rounded to fp32.
    const int half = s->D / 2;
    std::vector<float> ct((size_t)c.max_context * half), st((size_t)c.max_context * half);
    for (int p = 0; p < c.max_context; ++p)
        for (int i = 0; i < half; ++i) {
            const double ang = (double)p * std::pow((double)c.rope_theta, -2.0 * i / s->D);
            ct[(size_t)p * half + i] = (float)std::cos(ang);
            st[(size_t)p * half + i] = (float)std::sin(ang);
        }
    // on the compute stream and waited for: the stage's kernels run on non-blocking streams, which do
    // not wait for work on the null stream
    if (hipMemcpyAsync(s->d_cos, ct.data(), ct.size() * sizeof(float), hipMemcpyHostToDevice, s->cs) != hipSuccess ||
        hipMemcpyAsync(s->d_sin, st.data(), st.size() * sizeof(float), hipMemcpyHostToDevice, s->cs) != hipSuccess ||
        hipStreamSynchronize(s->cs) != hipSuccess)
        return cleanup(STAGE_EHIP);
    *out = s;
    return STAGE_OK;
}

int stage_destroy(stage *s) {
    if (!s) return STAGE_OK;
    DeviceGuard dg(s->cfg.device);
    if (s->cs) (void)hipStreamSynchronize(s->cs);
    if (s->xs) (void)hipStreamSynchronize(s->xs);
    for (LaneState &ln : s->lanes)
        if (ln.cs) (void)hipStreamSynchronize(ln.cs);
    for (Layer &l : s->layers)
        for (Block &k : l.blk) free_block(k);
    for (void *p : s->slots) (void)hipFree(p);
    for (auto &v : s->slot_ready)
        for (hipEvent_t e : v) (void)hipEventDestroy(e);
    for (hipEvent_t e : s->slot_free) (void)hipEventDestroy(e);
    for (TimeRec &r : s->recs) {
        if (r.a) (void)hipEventDestroy(r.a);
        if (r.b) (void)hipEventDestroy(r.b);
    }
    for (hipEvent_t e : s->ev_pool) (void)hipEventDestroy(e);
    for (hipEvent_t e : s->ready_ev)
        if (e) (void)hipEventDestroy(e);
    s->block_park.clear();
    for (void *p : s->park_host)
        if (p) (void)hipHostFree(p);
    for (void *p : {(void *)s->kv_pool, (void *)s->d_table, (void *)s->d_meta, (void *)s->d_cos, (void *)s->d_sin,
                    (void *)s->ws_qkv, (void *)s->ws_q, (void *)s->ws_attn, (void *)s->ws_h,
                    (void *)s->ws_pair,
                    (void *)s->ws_part_o, (void *)s->ws_part_ml, (void *)s->ws_split, (void *)s->ws_split_ss,
                    s->ws_dense, (void *)s->d_slot_tags, (void *)s->d_slot_rec})
        if (p) (void)hipFree(p);
    if (s->own_cs && s->cs) (void)hipStreamDestroy(s->cs);
    if (s->own_xs && s->xs) (void)hipStreamDestroy(s->xs);
    for (LaneState &ln : s->lanes) {
        for (void *p : {(void *)ln.d_meta, (void *)ln.ws_qkv, (void *)ln.ws_q, (void *)ln.ws_attn, (void *)ln.ws_h,
                        (void *)ln.ws_pair, (void *)ln.ws_part_o, (void *)ln.ws_part_ml,
                        (void *)ln.ws_split, (void *)ln.ws_split_ss})
            if (p) (void)hipFree(p);
        if (ln.own_cs && ln.cs) (void)hipStreamDestroy(ln.cs);
    }
    for (hipEvent_t e : s->seq_ev)
        if (e) (void)hipEventDestroy(e);
    delete s;
    return STAGE_OK;
}

int stage_load_layer(stage *s, int32_t layer, const stage_layer_weights *w, int32_t resident) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    if (layer < 0 || layer >= s->L || resident < STAGE_RES_OFFLOADED || resident > STAGE_RES_MLP_OFFLOADED)
        return s->fail(STAGE_EINVAL, "bad layer %d or residency %d", layer, resident);
    DeviceGuard dg(s->cfg.device);
    Layer &ly = s->layers[layer];
    if (!w) {
        if (!ly.loaded) return s->fail(STAGE_ESTATE, "layer %d was never loaded", layer);
        int rc = set_residency(s, layer, resident);
        if (rc == STAGE_OK) s->base_code[layer] = resident;
        return rc;
    }
    const void *src[9] = {w->wq, w->wk, w->wv, w->wo, w->wg, w->wu, w->wd, w->g1, w->g2};
    for (const void *p : src)
        if (!p) return s->fail(STAGE_EINVAL, "null weight pointer");
    int rc = check_residency(s, layer, resident);
    if (rc) return rc;
    Block fresh[2];
    for (int b = 0; b < 2; ++b) {
        rc = alloc_block(s, b, code_keeps(resident, b), &fresh[b]);
        if (rc) {
            free_block(fresh[0]);
            return rc;
        }
    }
    rc = sync_all(s);
    if (rc) {
        for (Block &k : fresh) free_block(k);
        return rc;
    }
    const size_t H = s->H, F = s->F, qd = (size_t)s->Hq * s->D, kvd = (size_t)s->Hkv * s->D;
    const int blk_of[9] = {kMha, kMha, kMha, kMha, kMlp, kMlp, kMlp, kMha, kMlp};
    const size_t offs[9] = {s->off_wqkv, s->off_wqkv + qd * H * 2, s->off_wqkv + (qd + kvd) * H * 2,
                            s->off_wo, s->off_wg, s->off_wu, s->off_wd, s->off_g1, s->off_g2};
    const size_t bytes[9] = {qd * H * 2, kvd * H * 2, kvd * H * 2, H * qd * 2, F * H * 2,
                             F * H * 2, H * F * 2, H * 2, H * 2};
    // Copies on the compute stream, then waited for: a device-to-device hipMemcpy on the null stream
    // returns before it completes, and kernels on a non-blocking compute stream would not wait for it
    // (they could read a half-copied layer).
    hipError_t e = hipSuccess;
    for (int i = 0; i < 9 && e == hipSuccess; ++i) {
        const Block &k = fresh[blk_of[i]];
        char *dst = static_cast<char *>(k.resident ? k.dev : k.host);
        e = hipMemcpyAsync(dst + offs[i], src[i], bytes[i], hipMemcpyDefault, s->cs);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(s->cs);
    if (e != hipSuccess) {
        for (Block &f : fresh) free_block(f);
        return s->fail_hip(e, "copying layer weights");
    }
    for (int b = 0; b < 2; ++b) {
        free_block(ly.blk[b]);
        ly.blk[b] = fresh[b];
    }
    ly.loaded = true;
    s->base_code[layer] = resident;
    return STAGE_OK;
}

int stage_prefill(stage *s, int32_t n_mb, const int32_t *mb_ids, int32_t B, int32_t T, const float *x_in,
                  float *x_out) {
    return run_call(s, n_mb, mb_ids, B, T, x_in, x_out, false);
}

int stage_decode(stage *s, int32_t n_mb, const int32_t *mb_ids, int32_t B, const float *x_in, float *x_out) {
    return run_call(s, n_mb, mb_ids, B, 1, x_in, x_out, true);
}

namespace {
// A call on decode lane `lane` >= 1 (stage_decode_lane, stage_prefill_lane).
static int run_lane_call(stage *s, int lane, int n_mb, const int32_t *mb_ids, int B, int T, const float *x_in, float *x_out,
                  bool decode) {
    if (lane < 0 || lane >= (int)s->lanes.size())
        return s->fail(STAGE_EINVAL, "lane %d out of range (%d lanes)", lane, std::max<int>(1, (int)s->lanes.size()));
    // a lane call stages no layer through the slots and moves no parked tail: both use the copy
    // stream and slot events that order the stage's calls one after another
    const bool direct = s->cfg.zero_copy && T == 1;
    for (int l = 0; l < s->L; ++l)
        if (s->layers[l].streams() && !direct)
            return s->fail(STAGE_ESTATE, "layer %d streams through the slots: lanes need resident (or zero-copy) layers", l);
    if (s->cfg.plan_mode || s->thresholds_applied < s->cfg.n_thresholds)
        return s->fail(STAGE_ESTATE, "a residency schedule is pending: lanes need a fixed residency");
    if (n_mb >= 1 && n_mb <= s->cfg.max_microbatches && mb_ids && B >= 1 && B <= s->cfg.max_batch)
        for (int k = 0; k < n_mb; ++k)
            for (int b = 0; b < B; ++b) {
                const int mb = mb_ids[k];
                if (mb < 0 || mb >= s->cfg.max_microbatches) continue;  // run_call reports it
                const int sl = seq_slot(s, mb, b);
                if (s->parked[sl] || s->ready_pending[sl])
                    return s->fail(STAGE_ESTATE, "micro-batch %d has a parked KV tail: run it on lane 0", mb);
            }
    swap_lane(s, lane);
    const int32_t timing = s->cfg.timing;
    s->cfg.timing = 0;  // events of lane calls are not recorded
    const int rc = run_call(s, n_mb, mb_ids, B, T, x_in, x_out, decode);
    s->cfg.timing = timing;
    swap_lane(s, lane);
    return rc;
}
}  // namespace

int stage_decode_lane(stage *s, int32_t lane, int32_t n_mb, const int32_t *mb_ids, int32_t B, const float *x_in,
                      float *x_out) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    if (lane == 0) return stage_decode(s, n_mb, mb_ids, B, x_in, x_out);
    return run_lane_call(s, lane, n_mb, mb_ids, B, 1, x_in, x_out, true);
}

int stage_prefill_lane(stage *s, int32_t lane, int32_t n_mb, const int32_t *mb_ids, int32_t B, int32_t T,
                       const float *x_in, float *x_out) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    if (lane == 0) return stage_prefill(s, n_mb, mb_ids, B, T, x_in, x_out);
    return run_lane_call(s, lane, n_mb, mb_ids, B, T, x_in, x_out, false);
}


int stage_decode_noalloc(stage *s, int32_t n_mb, const int32_t *mb_ids, int32_t B, const float *x_in,
                         float *x_out) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    const stage_config &c = s->cfg;
    if (n_mb < 1 || n_mb > c.max_microbatches || !mb_ids || B < 1 || B > c.max_batch || !x_in || !x_out)
        return s->fail(STAGE_EINVAL, "bad call arguments (n_mb=%d B=%d)", n_mb, B);
    std::vector<int> slots;
    std::vector<char> seen(c.max_microbatches, 0);
    for (int k = 0; k < n_mb; ++k) {
        const int mb = mb_ids[k];
        if (mb < 0 || mb >= c.max_microbatches || seen[mb])
            return s->fail(STAGE_EINVAL, "micro-batch id %d out of range or repeated", mb);
        seen[mb] = 1;
        for (int b = 0; b < B; ++b) slots.push_back(seq_slot(s, mb, b));
    }
    int longest = 0, max_after = 1;
    long long held = (long long)slots.size();
    for (int len : s->lengths) {
        longest = std::max(longest, len);
        held += len;
    }
    for (int sl : slots) {
        if (s->parked[sl]) return s->fail(STAGE_ESTATE, "sequence slot %d has a parked KV tail", sl);
        longest = std::max(longest, s->lengths[sl] + 1);
        max_after = std::max(max_after, s->lengths[sl] + 1);
    }
    const int splits = std::min(s->max_splits, (max_after + kDecodeSplitKeys - 1) / kDecodeSplitKeys);
    const ScratchLayout lay = scratch_layout(s, slots.size(), splits);
    if (lay.total > kScratchBytes)
        return s->fail(STAGE_ENOMEM, "the call needs %zu bytes of scratch; the limit is %zu (STAGE_NOALLOC_SCRATCH_BYTES)",
                       lay.total, kScratchBytes);
    // nothing in the call may allocate: no residency change, no first slot allocation
    if (c.plan_mode) {
        const std::vector<int> codes = plan_codes(s, held);
        for (int l = 0; l < s->L; ++l)
            if (codes[l] != code_of(s->layers[l]))
                return s->fail(STAGE_ESTATE, "the planner would change layer %d's residency in this call", l);
    } else if (s->thresholds_applied < c.n_thresholds && c.thresholds[s->thresholds_applied] <= longest) {
        return s->fail(STAGE_ESTATE, "a residency threshold is reached in this call");
    }
    if (!c.zero_copy && s->slots.empty()) {
        bool may_stream = c.plan_mode ? c.n_thresholds > 0 : s->thresholds_applied < c.n_thresholds;
        for (const Layer &ly : s->layers) may_stream = may_stream || ly.streams();
        if (may_stream) return s->fail(STAGE_ESTATE, "stream slots are not allocated yet (run stage_decode once)");
    }
    if (!s->scratch) return s->fail(STAGE_ESTATE, "no scratch array on this device");
    char *base = static_cast<char *>(s->scratch);
    LaneState ws;
    ws.d_meta = reinterpret_cast<CallMeta *>(base + lay.meta);
    ws.ws_rows = slots.size();
    ws.part_rows = slots.size();
    ws.ws_q = reinterpret_cast<float *>(base + lay.q);
    ws.ws_attn = reinterpret_cast<float *>(base + lay.attn);
    ws.ws_h = reinterpret_cast<float *>(base + lay.h);
    ws.ws_part_o = reinterpret_cast<float *>(base + lay.part_o);
    ws.ws_part_ml = reinterpret_cast<float *>(base + lay.part_ml);
    ws.ws_split = lay.has_split ? reinterpret_cast<float *>(base + lay.split) : nullptr;
    ws.ws_split_ss = lay.has_split ? reinterpret_cast<float *>(base + lay.split_ss) : nullptr;
    DeviceGuard dg(c.device);
    swap_workspaces(s, ws);
    const int saved_splits = s->max_splits;
    const int32_t timing = s->cfg.timing;
    s->max_splits = splits;  // the stride of the attention partials in the scratch array
    s->cfg.timing = 0;       // no timing events: their pool may have to create one
    const int rc = run_call(s, n_mb, mb_ids, B, 1, x_in, x_out, true);
    s->cfg.timing = timing;
    s->max_splits = saved_splits;
    swap_workspaces(s, ws);
    return rc;
}

int stage_kv_append(stage *s, int32_t mb, int32_t b, int32_t n_tokens, const void *k, const void *v) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    if (mb < 0 || mb >= s->cfg.max_microbatches || b < 0 || b >= s->cfg.max_batch || n_tokens < 1 || !k || !v)
        return s->fail(STAGE_EINVAL, "bad kv_append arguments");
    const int slot = seq_slot(s, mb, b);
    if (s->lengths[slot] + s->parked[slot] + n_tokens > s->cfg.max_context)
        return s->fail(STAGE_ERANGE, "sequence would exceed max_context");
    if (blocks_needed(s, slot, s->parked[slot] + n_tokens) > (int)s->free_blocks.size())
        return s->fail(STAGE_ENOMEM, "KV pool exhausted");
    DeviceGuard dg(s->cfg.device);
    if (int rc_ = join_lanes(s)) return rc_;
    const size_t elem = s->cfg.kv_fp32 ? 4 : 2;
    const size_t bytes = (size_t)s->L * n_tokens * s->Hkv * s->D * elem;
    const bool dev = is_device_ptr(k) && is_device_ptr(v);
    if (!dev) {
        int rc = ensure_dense(s, 2 * bytes);
        if (rc) return rc;
    }
    int rc = prepare_sequences(s, {slot});
    if (rc) return rc;
    rc = allocate_blocks(s, {slot}, n_tokens);
    if (rc) return rc;
    KvCopyArgs a = kv_copy_args(s, slot, s->lengths[slot], n_tokens, s->ws_dense, true);
    if (dev) {
        a.k = const_cast<void *>(k);
        a.v = const_cast<void *>(v);
    } else {
        HIP_TRY(hipMemcpyAsync(a.k, k, bytes, hipMemcpyHostToDevice, s->cs));
        HIP_TRY(hipMemcpyAsync(a.v, v, bytes, hipMemcpyHostToDevice, s->cs));
    }
    HIP_TRY(launch_kv_copy(a, s->cs));
    s->lengths[slot] += n_tokens;
    HIP_TRY(hipStreamSynchronize(s->cs));
    return STAGE_OK;
}

int stage_kv_export_tail(stage *s, int32_t mb, int32_t b, int32_t n_tokens, void *k, void *v, int32_t drop) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    if (mb < 0 || mb >= s->cfg.max_microbatches || b < 0 || b >= s->cfg.max_batch || n_tokens < 1 || !k || !v)
        return s->fail(STAGE_EINVAL, "bad kv_export_tail arguments");
    const int slot = seq_slot(s, mb, b);
    const int len = s->lengths[slot] + s->parked[slot];
    if (n_tokens > len) return s->fail(STAGE_ESTATE, "sequence holds %d tokens, %d requested", len, n_tokens);
    if (blocks_needed(s, slot, s->parked[slot]) > (int)s->free_blocks.size())
        return s->fail(STAGE_ENOMEM, "KV pool exhausted");
    DeviceGuard dg(s->cfg.device);
    if (int rc_ = join_lanes(s)) return rc_;
    const size_t elem = s->cfg.kv_fp32 ? 4 : 2;
    const size_t bytes = (size_t)s->L * n_tokens * s->Hkv * s->D * elem;
    const bool dev = is_device_ptr(k) && is_device_ptr(v);
    if (!dev) {
        int rc = ensure_dense(s, 2 * bytes);
        if (rc) return rc;
    }
    int rc = prepare_sequences(s, {slot});
    if (rc) return rc;
    KvCopyArgs a = kv_copy_args(s, slot, s->lengths[slot] - n_tokens, n_tokens, s->ws_dense, false);
    if (dev) {
        a.k = k;
        a.v = v;
    }
    HIP_TRY(launch_kv_copy(a, s->cs));
    if (!dev) {
        HIP_TRY(hipMemcpyAsync(k, a.k, bytes, hipMemcpyDeviceToHost, s->cs));
        HIP_TRY(hipMemcpyAsync(v, a.v, bytes, hipMemcpyDeviceToHost, s->cs));
    }
    HIP_TRY(hipStreamSynchronize(s->cs));
    if (drop) {
        s->lengths[slot] -= n_tokens;
        release_tail_blocks(s, slot);
    }
    return STAGE_OK;
}

int stage_reset_sequence(stage *s, int32_t mb, int32_t b) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    if (mb < 0 || mb >= s->cfg.max_microbatches || b < 0 || b >= s->cfg.max_batch)
        return s->fail(STAGE_EINVAL, "bad sequence (%d, %d)", mb, b);
    const int slot = seq_slot(s, mb, b);
    DeviceGuard dg(s->cfg.device);
    int rc = sync_all(s);  // freed blocks may be written by the copy stream without waiting for compute
    if (rc) return rc;
    s->lengths[slot] = 0;
    s->parked[slot] = 0;
    s->ready_pending[slot] = 0;
    release_tail_blocks(s, slot);
    return STAGE_OK;
}

int stage_kv_park(stage *s, int32_t n_mb, const int32_t *mb_ids, int32_t n_tokens) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    const stage_config &c = s->cfg;
    if (c.kv_park_tokens < 1) return s->fail(STAGE_ESTATE, "parking needs kv_park_tokens > 0");
    if (n_mb < 1 || n_mb > c.max_microbatches || !mb_ids || n_tokens < 1 || n_tokens > c.kv_park_tokens)
        return s->fail(STAGE_EINVAL, "bad kv_park arguments (n_mb=%d n_tokens=%d)", n_mb, n_tokens);
    std::vector<int> slots;
    std::vector<char> seen(c.max_microbatches, 0);
    for (int k = 0; k < n_mb; ++k) {
        const int mb = mb_ids[k];
        if (mb < 0 || mb >= c.max_microbatches || seen[mb])
            return s->fail(STAGE_EINVAL, "micro-batch id %d out of range or repeated", mb);
        seen[mb] = 1;
        for (int b = 0; b < c.max_batch; ++b) {
            const int sl = seq_slot(s, mb, b);
            if (s->parked[sl] > 0) return s->fail(STAGE_ESTATE, "sequence (%d, %d) is already parked", mb, b);
            if (s->lengths[sl] > 0) slots.push_back(sl);
        }
    }
    DeviceGuard dg(c.device);
    if (int rc_ = join_lanes(s)) return rc_;
    for (int sl : slots) {
        if (s->park_host[sl]) continue;
        void *hbuf = nullptr, *dbuf = nullptr;
        if (hipHostMalloc(&hbuf, 2 * tail_bytes(s, c.kv_park_tokens), hipHostMallocDefault) != hipSuccess) {
            (void)hipGetLastError();
            return s->fail(STAGE_ENOMEM, "pinned parking buffer of %zu bytes", 2 * tail_bytes(s, c.kv_park_tokens));
        }
        hipError_t e = hipHostGetDevicePointer(&dbuf, hbuf, 0);
        if (e != hipSuccess) {
            (void)hipHostFree(hbuf);
            return s->fail_hip(e, "hipHostGetDevicePointer");
        }
        s->park_host[sl] = hbuf;
        s->park_host_dev[sl] = dbuf;
    }
    if (slots.empty()) return STAGE_OK;
    auto done = std::make_shared<ParkEvent>();
    if (hipEventCreateWithFlags(&done->e, hipEventDisableTiming) != hipSuccess) {
        done->e = nullptr;
        return s->fail(STAGE_EHIP, "hipEventCreate failed");
    }
    hipEvent_t after = nullptr;
    int rc = record_event(s, s->cs, &after);  // the copies follow everything enqueued for compute
    if (rc) return rc;
    HIP_TRY(hipStreamWaitEvent(s->xs, after, 0));
    s->ev_pool.push_back(after);
    for (int sl : slots) {
        const int n = std::min(n_tokens, s->lengths[sl]);
        HIP_TRY(launch_kv_park(kv_park_args(s, sl, s->lengths[sl] - n, n, false), s->xs));
    }
    HIP_TRY(hipEventRecord(done->e, s->xs));
    for (int sl : slots) {
        const int n = std::min(n_tokens, s->lengths[sl]);
        s->lengths[sl] -= n;
        s->parked[sl] = n;
        release_tail_blocks(s, sl, done);
        s->bytes_parked += (long long)(2 * tail_bytes(s, n));
    }
    return STAGE_OK;
}

int stage_kv_unpark(stage *s, int32_t n_mb, const int32_t *mb_ids) {
    if (!s) return STAGE_EINVAL;
    s->err.clear();
    const stage_config &c = s->cfg;
    if (n_mb < 1 || n_mb > c.max_microbatches || !mb_ids) return s->fail(STAGE_EINVAL, "bad kv_unpark arguments");
    std::vector<int> slots;
    std::vector<char> seen(c.max_microbatches, 0);
    int need = 0;
    for (int k = 0; k < n_mb; ++k) {
        const int mb = mb_ids[k];
        if (mb < 0 || mb >= c.max_microbatches || seen[mb])
            return s->fail(STAGE_EINVAL, "micro-batch id %d out of range or repeated", mb);
        seen[mb] = 1;
        for (int b = 0; b < c.max_batch; ++b) {
            const int sl = seq_slot(s, mb, b);
            if (s->parked[sl] > 0) {
                slots.push_back(sl);
                need += blocks_needed(s, sl, s->parked[sl]);
            }
        }
    }
    if (need > (int)s->free_blocks.size())
        return s->fail(STAGE_ENOMEM, "KV pool exhausted (%d blocks needed, %d free)", need, (int)s->free_blocks.size());
    DeviceGuard dg(c.device);
    if (int rc_ = join_lanes(s)) return rc_;
    for (int sl : slots) {
        int rc = enqueue_unpark(s, sl);
        if (rc) return rc;
    }
    return STAGE_OK;
}

int stage_sync(stage *s) {
    if (!s) return STAGE_EINVAL;
    DeviceGuard dg(s->cfg.device);
    int rc = sync_all(s);
    if (rc) return rc;
    HIP_TRY(hipGetLastError());
    if (s->d_slot_rec) {
        int rec[8];
        HIP_TRY(hipMemcpy(rec, s->d_slot_rec, sizeof rec, hipMemcpyDeviceToHost));
        s->slot_checks_run += rec[0];
        if (rec[0] || rec[1]) {
            HIP_TRY(hipMemsetAsync(s->d_slot_rec, 0, sizeof rec, s->cs));
            HIP_TRY(hipStreamSynchronize(s->cs));
        }
        if (rec[1]) {
            static const char *const where[4] = {"before the MHA block's kernels", "before the MLP block's kernels",
                                                 "after the layer (MHA block)", "after the layer (MLP block)"};
            s->slot_check_failures += rec[1];
            return s->fail(STAGE_ESLOT,
                           "%d slot tag check(s) failed; first: slot %d %s expected layer %d load %d, found "
                           "layer %d load %d",
                           rec[1], rec[3], (rec[2] >= 0 && rec[2] < 4) ? where[rec[2]] : "?", rec[4], rec[5],
                           rec[6], rec[7]);
        }
    }
    return STAGE_OK;
}

int stage_get_block_table(stage *s, int32_t mb, int32_t b, int32_t *blocks, int32_t cap, int32_t *n) {
    if (!s || !n || cap < 0 || (cap > 0 && !blocks) || mb < 0 || mb >= s->cfg.max_microbatches || b < 0 ||
        b >= s->cfg.max_batch)
        return STAGE_EINVAL;
    const std::vector<int> &t = s->tables[seq_slot(s, mb, b)];
    *n = (int)t.size();
    for (int i = 0; i < std::min<int>(cap, (int)t.size()); ++i) blocks[i] = t[i];
    return STAGE_OK;
}

int stage_get_length(stage *s, int32_t mb, int32_t b, int32_t *length) {
    if (!s || !length || mb < 0 || mb >= s->cfg.max_microbatches || b < 0 || b >= s->cfg.max_batch)
        return STAGE_EINVAL;
    *length = s->lengths[seq_slot(s, mb, b)] + s->parked[seq_slot(s, mb, b)];
    return STAGE_OK;
}

int stage_get_residency(stage *s, int32_t *out) {
    if (!s || !out) return STAGE_EINVAL;
    for (int l = 0; l < s->L; ++l) out[l] = code_of(s->layers[l]);
    return STAGE_OK;
}

static int copy_log(const std::vector<int> &log, int width, int32_t *entries, int32_t cap, int32_t *n) {
    if (!n || cap < 0 || (cap > 0 && !entries)) return STAGE_EINVAL;
    const int count = (int)log.size() / width;
    *n = count;
    for (int i = 0; i < std::min<int>(cap, count) * width; ++i) entries[i] = log[i];
    return STAGE_OK;
}

int stage_get_slot_log(stage *s, int32_t *entries, int32_t cap, int32_t *n) {
    if (!s) return STAGE_EINVAL;
    return copy_log(s->slot_log, 3, entries, cap, n);
}

int stage_get_residency_log(stage *s, int32_t *entries, int32_t cap, int32_t *n) {
    if (!s) return STAGE_EINVAL;
    return copy_log(s->residency_log, 3, entries, cap, n);
}

int stage_get_demotion_log(stage *s, int32_t *entries, int32_t cap, int32_t *n) {
    if (!s) return STAGE_EINVAL;
    return copy_log(s->demotion_log, 2, entries, cap, n);
}

int stage_get_timeline(stage *s, float *records, int32_t cap, int32_t *n) {
    if (!s || !n || cap < 0 || (cap > 0 && !records)) return STAGE_EINVAL;
    DeviceGuard dg(s->cfg.device);
    int rc = sync_all(s);
    if (rc) return rc;
    *n = (int)s->recs.size();
    if (!s->recs.empty()) {
        // origin: the earliest start among the records
        std::vector<float> start(s->recs.size()), end(s->recs.size());
        for (size_t i = 0; i < s->recs.size(); ++i) {
            HIP_TRY(hipEventElapsedTime(&start[i], s->recs[0].a, s->recs[i].a));
            HIP_TRY(hipEventElapsedTime(&end[i], s->recs[0].a, s->recs[i].b));
        }
        const float t0 = *std::min_element(start.begin(), start.end());
        for (int i = 0; i < std::min<int>(cap, (int)s->recs.size()); ++i) {
            records[4 * i + 0] = (float)s->recs[i].kind;
            records[4 * i + 1] = (float)s->recs[i].layer;
            records[4 * i + 2] = start[i] - t0;
            records[4 * i + 3] = end[i] - t0;
        }
    }
    for (TimeRec &r : s->recs) {
        s->ev_pool.push_back(r.a);
        s->ev_pool.push_back(r.b);
    }
    s->recs.clear();
    return STAGE_OK;
}

int stage_set_timing(stage *s, int32_t flags) {
    if (!s || (flags & ~kTimeAll) != 0) return STAGE_EINVAL;
    s->cfg.timing = flags;
    return STAGE_OK;
}

int stage_get_stats(stage *s, char *buf, int32_t cap) {
    if (!s || !buf || cap < 1) return STAGE_EINVAL;
    int res = 0, streamed = 0, off_mha = 0, off_mlp = 0;
    size_t host_w = 0;
    long long parked = 0;
    for (int p : s->parked) parked += p;
    for (const Layer &l : s->layers) {
        if (!l.loaded) continue;
        for (int b = 0; b < 2; ++b) host_w += l.blk[b].host ? s->blk_bytes[b] : 0;
        res += code_of(l) == STAGE_RES_RESIDENT;
        streamed += l.streams();
        off_mha += !l.blk[kMha].resident;
        off_mlp += !l.blk[kMlp].resident;
    }
    const size_t hbm_w = resident_bytes(s) + s->slots.size() * s->blob_bytes;
    const int written = snprintf(
        buf, cap,
        "{\"calls\": %lld, \"prefill_tokens\": %lld, \"decode_tokens\": %lld, \"layer_loads\": %lld, "
        "\"bytes_streamed\": %lld, \"bytes_direct\": %lld, \"layer_bytes\": %zu, \"mha_block_bytes\": %zu, "
        "\"mlp_block_bytes\": %zu, \"resident_layers\": %d, \"streamed_layers\": %d, "
        "\"offloaded_mha_blocks\": %d, \"offloaded_mlp_blocks\": %d, "
        "\"stream_slots\": %zu, \"hbm_weight_bytes\": %zu, \"host_weight_bytes\": %zu, \"kv_pool_bytes\": %zu, "
        "\"kv_blocks\": %d, \"kv_blocks_free\": %d, \"parked_tokens\": %lld, \"bytes_parked\": %lld, "
        "\"bytes_unparked\": %lld, \"kernel_launches\": %lld, \"last_call_kernels\": %lld, "
        "\"slot_check\": %d, \"slot_checks\": %lld, \"slot_checks_run\": %lld, \"slot_check_failures\": %lld}",
        s->calls, s->tok_prefill, s->tok_decode, s->loads, s->bytes_streamed, s->bytes_direct, s->blob_bytes,
        s->blk_bytes[kMha], s->blk_bytes[kMlp], res, streamed, off_mha, off_mlp,
        s->slots.size(), hbm_w, host_w, s->kv_layer_stride * s->L, s->n_blocks, (int)s->free_blocks.size(),
        parked, s->bytes_parked, s->bytes_unparked, s->kernel_launches, s->last_call_kernels, s->cfg.slot_check,
        s->slot_checks, s->slot_checks_run, s->slot_check_failures);
    return (written >= 0 && written < cap) ? STAGE_OK : STAGE_EINVAL;
}

}  // extern "C"
