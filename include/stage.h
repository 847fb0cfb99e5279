/*
 * stage.h -- C ABI of one pipeline stage of the offloading-based interleaved
 * pipeline (arXiv 2512.21835), on one MI355X (gfx950) GPU.
 *
 * A stage is a contiguous block of LLaMA-style decoder layers (Section III-A:
 * every device holds stages of consecutive layers and runs micro-batches
 * through them in turn).  Some layers are *resident* in HBM; the others are
 * *offloaded* to pinned host memory and streamed, layer by layer, into a few
 * reusable HBM slots while resident layers compute (Section III-A: retained and
 * offloaded layers per stage; Section III-B: weight memory is the retained
 * layers plus one stage's worth of offloaded layers; Section III-C: a reusable
 * loading buffer refilled once the GPU signals it has finished with it).
 * Residency is per block: a layer's MHA block (Wq, Wk, Wv, Wo, g1) and its MLP
 * block (Wg, Wu, Wd, g2) can be resident or offloaded independently (Section
 * III-D, block-level offloading).
 * Streaming changes where the weights are, never the arithmetic: outputs are
 * bit-identical whichever layers are resident (lossless inference, abstract and
 * Section IV-A).
 *
 * Conventions for every function:
 *  - Return 0 (STAGE_OK) or a negative stage_status.  Nothing throws or aborts.
 *  - All arguments are validated before any state changes; on an error the
 *    handle is unchanged and still usable (except STAGE_EHIP, see below).
 *  - STAGE_EHIP reports a failed HIP call, possibly an asynchronous error of
 *    earlier work surfacing now; stage_last_error() gives the HIP message.
 *  - A handle is not thread-safe: use it from one host thread at a time.
 *  - Compute is enqueued on the compute stream and returns before it runs,
 *    unless stated otherwise.  Device buffers passed in must stay valid until
 *    the compute stream has passed the call (stage_sync or a stream sync).
 *  - Matrices are row-major.  Weights are [out, in] (each output row is
 *    contiguous).  bf16 is passed as its 16-bit pattern.
 *  - Sequences are addressed by (micro-batch id mb, batch row b), 0 <= mb <
 *    max_microbatches, 0 <= b < max_batch.  Each has its own KV cache and
 *    positions; a sequence starts empty and its positions continue from its
 *    current length.
 */
#ifndef PAPER_2512_21835_STAGE_H
#define PAPER_2512_21835_STAGE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct stage stage; /* opaque; one per stage per GPU */

typedef enum {
    STAGE_OK = 0,
    STAGE_EINVAL = -1, /* bad argument */
    STAGE_ENOMEM = -2, /* HBM budget, device/pinned allocation or KV block pool exhausted */
    STAGE_EHIP = -3,   /* a HIP runtime call failed */
    STAGE_ESTATE = -4, /* not valid now (layer not loaded, sequence empty, ...) */
    STAGE_ERANGE = -5, /* a sequence would exceed max_context */
    STAGE_ESLOT = -6   /* a slot tag check failed (stage_config.slot_check; reported by stage_sync) */
} stage_status;

#define STAGE_MAX_THRESHOLDS 32
#define STAGE_MAX_SEQS_PER_CALL 64
#define STAGE_MAX_CONTEXT 16384
#define STAGE_MAX_LANES 4

/* Residency of a layer (stage_load_layer, stage_get_residency).  "MHA-only offloading" in the
   sense of Section III-D: the MHA block streams, the MLP block stays resident. */
#define STAGE_RES_OFFLOADED 0      /* both blocks in pinned host memory */
#define STAGE_RES_RESIDENT 1       /* both blocks in HBM */
#define STAGE_RES_MHA_OFFLOADED 2  /* MHA block offloaded, MLP block resident */
#define STAGE_RES_MLP_OFFLOADED 3  /* MLP block offloaded, MHA block resident */

/* Timing flags (stage_config.timing). */
#define STAGE_TIME_CALLS 1   /* events around each prefill/decode call and each slot copy */
#define STAGE_TIME_GATEUP 2  /* events around the gate/up projection kernel of one decode layer
                                per call (layer = call number mod n_layers) */
#define STAGE_TIME_LAYERS 4  /* events around each layer's MHA-block and MLP-block kernels */

typedef struct {
    /* Layer shape.  hidden, head_dim, ffn and n_q_heads*head_dim must be multiples of 8;
       head_dim even and <= 256; n_q_heads a multiple of n_kv_heads. */
    int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn;
    float rope_theta; /* RoPE base; angle of pair i at position p is p * theta^(-2i/head_dim) */
    float rms_eps;    /* RMSNorm epsilon, added to mean(x^2) inside the square root */
    /* Sequence capacity.  max_microbatches * max_batch <= STAGE_MAX_SEQS_PER_CALL;
       max_context <= STAGE_MAX_CONTEXT. */
    int32_t max_microbatches, max_batch, max_context;
    int32_t kv_block_tokens; /* tokens per KV block; must be 16 */
    int32_t kv_pool_blocks;  /* blocks in the pool; 0 = every sequence can reach max_context */
    int32_t kv_fp32;         /* KV element type: 0 = bf16 (rounded to nearest even), 1 = fp32 */
    /* Weight memory: resident blocks may hold at most n_resident_max whole layers' bytes of HBM
       (the HBM weight budget, in layers; a block counts its own bytes); every layer with an
       offloaded block streams through n_stream_slots reusable HBM slots of one layer each.  Without
       zero_copy the slots are allocated when the first layer is offloaded; with zero_copy, by the
       first call that stages a layer (n_stream_slots may then be 0 for a stage that only runs
       one-token calls; a call that would stage fails with EINVAL). */
    int32_t n_resident_max;
    int32_t n_stream_slots;
    /* Residency schedule (Section III-E, online memory-aware planner): before a prefill or
       decode call, every threshold not yet applied that is <= the longest sequence length
       the stage will hold after the call demotes one resident layer, highest id first.
       Ascending; n_thresholds <= STAGE_MAX_THRESHOLDS. */
    int32_t n_thresholds;
    int32_t thresholds[STAGE_MAX_THRESHOLDS];
    int32_t device;       /* HIP device ordinal */
    /* Streams.  NULL: the library creates the stream on a hardware queue of its own (a stream
       with a compute-unit mask that enables every compute unit; it waits for work on the null
       stream like any blocking stream).  HIP otherwise maps streams onto a few shared hardware
       queues in creation order, and a copy stream sharing the compute stream's queue serialises
       the slot copies with the kernels (Section III-A's loading under computation is lost), so a
       caller that passes copy_stream must give it a queue of its own; NULL is recommended. */
    void *compute_stream; /* hipStream_t for kernels */
    void *copy_stream;    /* hipStream_t for slot copies and KV parking */
    int32_t timing;       /* STAGE_TIME_* flags; 0 = no events */
    /* 0 (default): offloaded layers are copied into a stream slot before their kernels run.
       1: calls with one token per sequence (every decode call, and a prefill with T = 1) run the
       kernels of offloaded layers on the pinned host blob directly, read over the host link (the
       zero-copy access of Section III-C): no slot copy and no slot-log entry for them.  Longer
       prefills still stage through the slots, since their GEMMs re-read every weight tile.
       Outputs are identical in both modes. */
    int32_t zero_copy;
    /* Residency schedule mode.  0: the thresholds above (longest sequence; each offloads one more
       layer).  1: steps of the online memory-aware planner (Section III-E, Eq. (7); computed by
       stage_plan_offload, include/stage_planner.h): thresholds[j] counts the tokens the stage
       holds over all sequences once the call's tokens are appended, ascending from >= 0.  While
       it holds at least thresholds[j] tokens (and fewer than thresholds[j+1]), the plan_alpha[j]
       highest-id layers whose MHA block the loaded allocation keeps resident have it offloaded,
       and likewise plan_beta[j] MLP blocks (all of them if fewer); below thresholds[0] the
       allocation stands.  The allocation is the residency last set by stage_load_layer.  The plan
       follows the token count both ways: a cache that shrinks (stage_kv_export_tail with drop,
       stage_reset_sequence) reloads blocks at the next call. */
    int32_t plan_mode;
    int32_t plan_alpha[STAGE_MAX_THRESHOLDS];
    int32_t plan_beta[STAGE_MAX_THRESHOLDS];
    /* Most tokens stage_kv_park moves out per sequence (0 = parking off).  Sizes one pinned host
       buffer per parked sequence, 2 * n_layers * kv_park_tokens * n_kv_heads * head_dim KV
       elements, which the parking kernels read and write directly over the host link. */
    int32_t kv_park_tokens;
    /* Decode lanes (0 or 1: one).  Lane l (1 <= l < n_lanes) has its own stream and workspaces, so
       decode calls on different lanes (stage_decode_lane) run concurrently: the interleaved
       schedule's independent micro-batches, whose weight streams then fill each other's
       latency-bound phases.  lane_streams[l]: lane l's hipStream_t (NULL = the library creates
       one, as for the streams above); lane 0 is compute_stream. */
    int32_t n_lanes;
    void *lane_streams[STAGE_MAX_LANES];
    /* Slot tag check (Section III-C: a reusable slot is refilled only after the kernels reading
       its previous layer have finished, and read only after its copy completed).  0: off.
       1: each stream slot carries a tag per block (layer, load number of the stage's life).  The
       copy stream invalidates a block's tag before copying into it and writes the new tag after
       the copy; on the compute stream a one-thread kernel compares the tag with the layer and load
       the call expects before the block's first kernel and again after the layer's last kernel,
       and counts mismatches in device memory.  A mismatch before means the block was not (or not
       yet) loaded; after, that the copy stream started refilling the slot while the layer still
       read it.  stage_sync returns STAGE_ESLOT once any check has failed since the previous
       stage_sync (stage_last_error names the first mismatch) and clears the count.  Costs one
       check kernel per streamed block before and after its layer and two tag writes per copy;
       outputs are bit-identical to mode 0.  2: as 1, but the checks before MHA blocks expect the
       next load number, so that they fail: a self-test of the detection path that changes no
       weight and no output. */
    int32_t slot_check;
} stage_config;

/* Weights of one decoder layer: bf16 bit patterns, host or device memory, read only during
   the call.  wq [Hq*d, H], wk [Hkv*d, H], wv [Hkv*d, H], wo [H, Hq*d], wg [F, H], wu [F, H],
   wd [H, F], g1 [H] (attention RMSNorm gain), g2 [H] (MLP RMSNorm gain). */
typedef struct {
    const void *wq, *wk, *wv, *wo, *wg, *wu, *wd, *g1, *g2;
} stage_layer_weights;

/* Fills *cfg with defaults: theta 10000, eps 1e-5, kv_block_tokens 16, n_stream_slots 2,
   device 0, everything else zero. */
void stage_config_default(stage_config *cfg);

/* Creates a stage on cfg->device.  Allocates the KV pool, the block tables and the
   RoPE tables in HBM.  No layer is loaded yet.
   EINVAL: inconsistent shape or capacity; ENOMEM: the KV pool does not fit; EHIP. */
int stage_init(const stage_config *cfg, stage **out);

/* Frees everything the stage owns after waiting for its streams.  NULL is a no-op. */
int stage_destroy(stage *s);

/* Loads layer `layer` (0 <= layer < n_layers) and sets its residency `resident`, a STAGE_RES_*
   code (Section III-A: retained vs offloaded layers; Section III-D: MHA or MLP block only).
   w != NULL: copy the weights into library storage -- HBM for a resident block, pinned host
   memory (hipHostMalloc) for an offloaded one; device sources must hold their values when the
   call is made (e.g. written on the compute stream); the copies run on the compute stream and the
   call waits for them, so the caller may free w on return.  w == NULL: change the residency of an already loaded layer (each
   block that changes side is copied across), which is the planner's offload action (Section
   III-E).  EINVAL: bad layer or code; ENOMEM: the resident blocks would exceed the weight budget,
   or allocation failed (the layer is unchanged); ESTATE: w == NULL for a layer never loaded. */
int stage_load_layer(stage *s, int32_t layer, const stage_layer_weights *w, int32_t resident);

/* Prefill: runs T new tokens of each of B rows of each listed micro-batch through all layers.
   x_in, x_out: device fp32 [n_mb][B][T][hidden] (x_out may not alias x_in).  Row r of x_out is
   the hidden state after the stage's last layer (no final norm).  The k-th micro-batch of the
   call is mb_ids[k] (distinct).  Streamed layers are loaded once per call, in ascending order,
   and run for all rows of the call before their slot is reused (Section III-A: loading
   overlapped with computation of other layers; the bursty pattern serves several micro-batches
   per load).  KV blocks are taken in call order (mb_ids order, then b ascending).
   EINVAL: bad ids/sizes or a layer not loaded; ERANGE: a sequence would exceed max_context;
   ENOMEM: KV pool exhausted. */
int stage_prefill(stage *s, int32_t n_mb, const int32_t *mb_ids, int32_t B, int32_t T,
                  const float *x_in, float *x_out);

/* Decode: one new token for each of B rows of each listed micro-batch; x_in, x_out: device
   fp32 [n_mb][B][hidden].  Same rules as stage_prefill with T = 1.  Every listed sequence
   must already hold at least one token (ESTATE otherwise). */
int stage_decode(stage *s, int32_t n_mb, const int32_t *mb_ids, int32_t B, const float *x_in,
                 float *x_out);

/* stage_decode on decode lane `lane` (0 <= lane < n_lanes; lane 0 is stage_decode itself): the
   call runs on the lane's stream with its workspaces, so calls on different lanes may overlap on
   the GPU.  A call waits (on the GPU) for the last call on another lane that touched any of its
   sequences, so a sequence's steps stay in order whichever lanes they use (stage_prefill and
   stage_decode order themselves the same way); the caller orders the call's inputs and outputs
   with the lane's stream.  The KV entry points (append, export, park, unpark, reset) and
   stage_load_layer synchronize all lanes first.  ESTATE for lanes >= 1 when a layer would be staged through the
   slots (lanes need resident or zero-copy layers), a residency schedule is pending, or a
   sequence of the call has a parked KV tail; EINVAL for a lane out of range; otherwise as
   stage_decode.  Outputs are identical to stage_decode's. */
int stage_decode_lane(stage *s, int32_t lane, int32_t n_mb, const int32_t *mb_ids, int32_t B, const float *x_in,
                      float *x_out);

/* stage_prefill on lane `lane`, with the same rules as stage_decode_lane: a new request's prefill
   can overlap other micro-batches' decode calls (its matrix-core GEMMs against their weight
   streams).  Outputs are identical to stage_prefill's. */
int stage_prefill_lane(stage *s, int32_t lane, int32_t n_mb, const int32_t *mb_ids, int32_t B, int32_t T,
                       const float *x_in, float *x_out);

/* Size of the per-GPU scratch array used by stage_decode_noalloc: 64 MiB. */
#define STAGE_NOALLOC_SCRATCH_BYTES 67108864

/* stage_decode for callers that cannot allocate device memory during the call (code under HIP
   graph capture, tight serving loops, harnesses that forbid hipMalloc): the same kernels and the
   same outputs as stage_decode, with their workspaces (row metadata, rotated queries, attention
   split partials and output, SwiGLU output, split-K partials) carved out of one fixed scratch
   array that every GPU the library runs on holds from the library's load until the process ends
   (STAGE_NOALLOC_SCRATCH_BYTES; its device address is looked up once per device by stage_init).
   The call makes no hipMalloc, hipFree or other allocating call and records no timing events.
   Every call on one GPU shares that GPU's array and leaves its contents behind: calls that
   overlap on one GPU (other stages' noalloc calls on other streams, or this stage's on other
   lanes) race; calls ordered on one stream are safe.  The caller still owns x_in and x_out.
   ENOMEM: the call needs more scratch than the array holds (the message gives the bytes; it
   grows with rows x (2 Hq d + ffn) and rows x Hq x ceil(context / 64) x (d + 2), plus a split-K
   area for 3 rows or more); ESTATE: the call would allocate -- a residency change is due (the
   threshold schedule or the planner), stream slots have not been allocated yet (run one
   stage_decode first), or a sequence of the call has a parked KV tail; otherwise as
   stage_decode.  Nothing changes on an error. */
int stage_decode_noalloc(stage *s, int32_t n_mb, const int32_t *mb_ids, int32_t B, const float *x_in,
                         float *x_out);

/* Appends n_tokens positions of already-rotated K and V to sequence (mb, b) without compute:
   the concatenation of a received KV-cache tail in the KV transfer protocol (Section III-E,
   Alg. 2).  k, v: [n_layers][n_tokens][n_kv_heads][head_dim] in the KV element type (bf16 bits
   or fp32), host or device memory; the call returns once they have been read.
   ERANGE / ENOMEM as for prefill. */
int stage_kv_append(stage *s, int32_t mb, int32_t b, int32_t n_tokens, const void *k,
                    const void *v);

/* Copies the stored K and V of the last n_tokens positions of sequence (mb, b) into k, v
   (layout and type as stage_kv_append; host or device memory; synchronous), and if drop != 0
   removes them from the sequence, returning emptied blocks to the pool: the tail a device ships
   to its peer in Alg. 2 (Section III-E).  ESTATE: fewer than n_tokens stored. */
int stage_kv_export_tail(stage *s, int32_t mb, int32_t b, int32_t n_tokens, void *k, void *v,
                         int32_t drop);

/* Forgets sequence (mb, b): its blocks return to the pool, a parked tail is dropped and its length
   becomes 0.  Waits for both streams. */
int stage_reset_sequence(stage *s, int32_t mb, int32_t b);

/* KV transfer protocol, the single-GPU half (Section III-E, Alg. 2: a device ships the tail of a
   stage's cache away after the stage runs and receives it back before the stage runs again),
   with pinned host memory as the peer.  Between two calls of a micro-batch its tails need no
   HBM, so the pool serves more sequences, and the copies overlap other micro-batches' compute.

   stage_kv_park enqueues on the copy stream, after all work enqueued so far on the compute
   stream, the move of the last min(n_tokens, length) tokens of every sequence of the listed
   micro-batches into pinned host memory, and returns their emptied blocks to the pool at once
   (compute-stream work enqueued later waits for these copies before it can write a block).
   A sequence keeps its length (stage_get_length counts parked tokens); its block table shrinks.
   The residency schedules count only tokens in HBM.  Returns before the copies run.
   1 <= n_tokens <= kv_park_tokens.  ESTATE: parking is off, or a listed sequence already has a
   parked tail; ENOMEM: the pinned buffer cannot be allocated (nothing changes). */
int stage_kv_park(stage *s, int32_t n_mb, const int32_t *mb_ids, int32_t n_tokens);

/* Enqueues on the copy stream the return of the listed micro-batches' parked tails into new
   blocks (taken lowest id first, sequence by sequence), without waiting for the compute stream,
   so that it overlaps compute already enqueued (the paper's asynchronous receive of the next
   stage's cache); the next compute on a returned sequence waits for its copy.  A call, append
   or export on a parked sequence returns its tail itself first.  Sequences without a parked
   tail are skipped.  ENOMEM: the pool lacks the blocks (nothing changes). */
int stage_kv_unpark(stage *s, int32_t n_mb, const int32_t *mb_ids);

/* Waits for the compute and copy streams; reports asynchronous HIP errors. */
int stage_sync(stage *s);

/* --- introspection (tests, metrics) --- */

/* Block ids of sequence (mb, b) in position order (block j holds positions 16j..16j+15);
   writes min(cap, count) ids, *n = count. */
int stage_get_block_table(stage *s, int32_t mb, int32_t b, int32_t *blocks, int32_t cap,
                          int32_t *n);

/* Current length of sequence (mb, b): tokens stored, in HBM or parked. */
int stage_get_length(stage *s, int32_t mb, int32_t b, int32_t *length);

/* Residency of every layer: a STAGE_RES_* code, -1 if not loaded; out has n_layers entries. */
int stage_get_residency(stage *s, int32_t *out);

/* Slot log: one (call number, layer, slot) triple per streamed-layer load (a layer with any
   offloaded block) since init, in load order; call numbers count prefill and decode calls from 0.
   Writes min(cap, count) triples (3*cap ints), *n = count. */
int stage_get_slot_log(stage *s, int32_t *entries, int32_t cap, int32_t *n);

/* Demotions made by the threshold schedule (plan_mode 0): (call number, layer) pairs, like the
   slot log.  A demotion offloads both blocks of the highest-id layer that still has a resident
   block. */
int stage_get_demotion_log(stage *s, int32_t *entries, int32_t cap, int32_t *n);

/* Every residency change made by the schedule, in either plan_mode: (call number, layer, new
   STAGE_RES_* code) triples in the order applied (within a call, ascending layer).  Writes
   min(cap, count) triples (3*cap ints), *n = count. */
int stage_get_residency_log(stage *s, int32_t *entries, int32_t cap, int32_t *n);

/* Timeline recorded under stage_config.timing, then cleared.  Synchronises.  Each record is
   four floats: kind (0 call, 1 slot copy of an MHA block, 2 gate/up kernel, 3 a layer's
   MHA-block kernels, 4 slot copy of an MLP block, 5 a layer's MLP-block kernels), layer (-1 for
   a call), start and end in milliseconds from the first record.  Kinds 3 and 5 exclude the wait
   for an MLP block still being copied.  Writes min(cap, count) records, *n = count. */
int stage_get_timeline(stage *s, float *records, int32_t cap, int32_t *n);

/* Replaces the STAGE_TIME_* flags of the stage (see stage_config.timing) for later calls. */
int stage_set_timing(stage *s, int32_t flags);

/* JSON object with counters: calls, tokens, layer loads, bytes streamed through slots and read in
   place (zero copy), block sizes, residency counts, HBM bytes in use, parked tokens and bytes
   moved by parking, kernels enqueued by prefill/decode calls in all and by the last one, and the
   slot tag checks enqueued, run and failed (the last two as of the latest stage_sync). */
int stage_get_stats(stage *s, char *buf, int32_t cap);

/* Message of the last error on this handle ("" if none); valid until the next call. */
const char *stage_last_error(stage *s);

/* Static description of a status code. */
const char *stage_strerror(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* PAPER_2512_21835_STAGE_H */
