/*
 * hisparse.h -- C ABI of the HiSparse decode hot path on AMD Instinct MI355X (gfx950).
 *
 * HiSparse ("Scaling Sparse-Attention Decoding with Hierarchical KV Cache Management") keeps
 * every request's full KV history in pinned host memory and gives each (request, layer) a
 * small fixed-size GPU cache of B record slots (Section 3.2). Each decode step, the sparse
 * indexer emits k selected logical records per request and layer; the library resolves them
 * against the cache -- hit detection, LRU victim choice among the slots this step does not
 * reference, fetch of the misses from pinned host memory into the freed HBM slots, and
 * emission of the physical slot of every selected record in the selection's order
 * (Section 3.4, phases 1-5) -- and then runs sparse decode attention over the k gathered
 * records. For models whose layers share one indexer's selection, the anchor layer's miss
 * plan is replayed into every shared layer's cache (Section 3.5, exact prefetch).
 *
 * Terms used below
 *   unit   one independent cache: a (request, layer) for token-level selection, or a
 *          (request, layer, kv head) for block/page selection. Unit u of a layer call is
 *          request * units_per_request + head.
 *   L      logical records per unit (tokens, blocks or pages), positions 0 .. L-1.
 *   R      bytes per record.   k  selected records per unit per step.   B  slots per unit.
 *
 * Conventions
 *   - Pointers prefixed d_ are device (HBM) pointers owned by the caller; the library reads or
 *     writes them on the given stream and keeps no reference after the call returns.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   - Calls marked [async] enqueue GPU work on `stream`, never synchronise the host, allocate
 *     nothing and can be captured in a HIP graph (with HISPARSE_FETCH_SDMA or
 *     HISPARSE_FETCH_STAGED, the calls that fetch synchronise `stream` once to read the miss
 *     plan back, and cannot be captured).
 *     Calls marked [sync] block the host.
 *   - Every call returns HISPARSE_OK or a negative hisparse_status_t; an argument error is
 *     reported before any work is enqueued, and leaves all state untouched.
 *   - Data errors found on the device (a selection entry >= L, or a repeated entry within one
 *     unit's selection) do not fail the enqueueing call: that unit's state is left unchanged,
 *     its k output slots are -1, its counts are (0, 0), and the error is latched for
 *     hisparse_check_errors. Negative selection entries are padding: output slot -1, not
 *     counted, never fetched.
 *   - One handle must not be used by two host threads at once; calls on one handle that touch
 *     the same layer must be ordered by the caller's streams.
 */
#ifndef HISPARSE_H
#define HISPARSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hisparse_cache* hisparse_cache_t;

typedef enum {
  HISPARSE_OK = 0,
  HISPARSE_ERR_INVALID_ARG = -1,   /* bad descriptor, layer index, pointer or size */
  HISPARSE_ERR_OOM = -2,           /* device or pinned host allocation failed */
  HISPARSE_ERR_HIP = -3,           /* a HIP runtime call failed */
  HISPARSE_ERR_UNSUPPORTED = -4,   /* valid request the library does not implement */
  HISPARSE_ERR_BAD_SELECTION = -5, /* latched device-side selection error (see above) */
  HISPARSE_ERR_FULL = -6           /* every request slot is taken (hisparse_request_acquire) */
} hisparse_status_t;

/* How missed records travel from the host pool to the GPU cache (Section 3.4 Phase 4). */
typedef enum {
  /* GPU threads load the missed records straight from mapped pinned host memory with 16-byte
   * vector loads and store them into their slots: the GPU-assisted IO the paper adopts. */
  HISPARSE_FETCH_ZERO_COPY = 0,
  /* The host reads the miss plan back (a stream synchronisation) and issues one batched DMA
   * copy (hipMemcpyBatchAsync) of the missed records. Not capturable in a HIP graph: calls
   * that fetch return HISPARSE_ERR_UNSUPPORTED while `stream` is capturing. */
  HISPARSE_FETCH_SDMA = 1,
  /* Timing mode (the no-IO oracle of Section 4.6): tables and slot outputs are exact, but no
   * record is copied, so the cache holds stale data and attention outputs are not valid. */
  HISPARSE_FETCH_NONE = 2,
  /* Staging DMA (the staging alternative to GPU-assisted IO, Section 3.4 Phase 4): the host reads
   * the miss plan back (a stream synchronisation), host threads gather the missed records from
   * the pool into a pinned staging buffer, one copy-engine transfer moves them to the device
   * and a kernel scatters them into their slots. Not capturable, like HISPARSE_FETCH_SDMA; the
   * cache also holds top_k * R bytes of pinned and of device staging memory per unit, which
   * its staged fetches share: each one first waits on the host until the previous one, on
   * whatever stream, has scattered out of them. */
  HISPARSE_FETCH_STAGED = 3
} hisparse_fetch_t;

/* Kind of pinned host memory backing the pool. */
typedef enum {
  HISPARSE_HOST_COHERENT = 0,      /* fine-grained, mapped (hipHostMallocCoherent|Mapped) */
  HISPARSE_HOST_NONCOHERENT = 1,   /* coarse-grained, mapped (hipHostMallocNonCoherent|Mapped) */
  HISPARSE_HOST_UNCACHED = 2       /* fine-grained uncached (hipHostMallocUncached|Mapped) */
} hisparse_host_memory_t;

/* Cache descriptor (the paper's configuration: top_k, device buffer size B, transfer block
 * size; Appendix A "Configuration", Section 3.2 "Sizing the cache"). */
typedef struct {
  int32_t num_requests;          /* >= 1 */
  int32_t num_layers;            /* >= 1 */
  int32_t units_per_request;     /* 1 (token-level) or kv heads (block/page selection) */
  int32_t capacity;              /* B: slots per unit; top_k <= B <= 16384 */
  int64_t num_records;           /* L: records per unit, 1 .. 2^31-1 */
  int32_t top_k;                 /* k: 1 .. 4096. The resolve kernel takes 16 * round_up(k, 4)
                                    + B / 4 + 8192 bytes of LDS (at most 76 KiB); create returns
                                    UNSUPPORTED on a device whose workgroups get less */
  int32_t record_bytes;          /* R: multiple of 16, 16 .. 1 MiB */
  int32_t share_group;           /* G >= 1: layers with layer % G == 0 are anchors that resolve;
                                    layer l with l % G != 0 shares the selection of anchor
                                    l - l % G (Section 3.5) */
  int32_t fetch;                 /* hisparse_fetch_t */
  int32_t host_memory;           /* hisparse_host_memory_t */
  int32_t transfer_block_bytes;  /* bytes each fetch thread keeps in flight: 16, 32, 64, 128
                                    or 256 (the paper's swap-in transfer block size); 0 = 16 */
  int32_t fetch_workgroups;      /* one-wave (64-thread) workgroups of one fetch launch,
                                    0 .. 4096, shared by its units and target layers (at least
                                    one per unit and layer); 0 = 192 for records under 4 KiB,
                                    256 for larger ones (measured best). A few hundred KB of host
                                    reads in flight saturate the link, so a thin grid moves
                                    misses as fast as a wide one while keeping few slow host
                                    reads outstanding per CU, which leaves kernels of other
                                    streams on the same CUs (attention, resolve) nearly
                                    undisturbed */
} hisparse_cache_desc_t;

/* Sparse decode attention descriptor. The token layout inside a record is
 * [tokens_per_record][token_elems] bf16 with token_elems = record_bytes / 2 / tokens_per_record;
 * the key is the token's first d_qk elements and the value its d_v elements from v_offset.
 * Supported shapes: (d_qk, d_v, v_offset) = (576, 512, 0), latent MLA where the value is the
 * first 512 dims of the 576-dim latent record; and (128, 128, 128), GQA with K then V.
 * top_k * tokens_per_record (tokens per unit) is at most 2^24, and at most 2^20 for latent MLA
 * (HISPARSE_ERR_UNSUPPORTED above that). */
typedef struct {
  int32_t q_heads;               /* query heads attending to one unit: 1 .. 256 */
  int32_t d_qk;
  int32_t d_v;
  int32_t v_offset;
  int32_t tokens_per_record;     /* 1 (token records), 16 (pages), 64 (blocks), ... */
  int32_t num_splits;            /* partitions of the token sequence reduced in a fixed order;
                                    0 = chosen from the shape alone */
  float scale;                   /* softmax scale applied to q.k */
  int32_t flags;                 /* 0 or HISPARSE_ATTN_DEFER_MERGE | HISPARSE_ATTN_BESIDE_FETCH |
                                    HISPARSE_ATTN_CARRIES_REPLAY */
} hisparse_attn_desc_t;

/* hisparse_attn_desc_t.flags: the attention call runs only its per-split workgroups (and any
 * replay it carries) and leaves the splits' partial results in d_workspace without writing
 * d_out; hisparse_attention_merge then writes d_out from them. For callers that schedule,
 * overlap or time the two kernels apart. */
#define HISPARSE_ATTN_DEFER_MERGE 1
/* hisparse_attn_desc_t.flags, a scheduling hint for latent attention: the call runs beside
 * another stream's host-link fetch (e.g. two micro-batches taking turns on the link), whose slow
 * host reads occupy the memory pipelines of the CUs they run on. The plan then aims at half a
 * workgroup per CU instead of one (fewer, longer splits): the fetch's waves find CUs without an
 * attention workgroup, and the split partial results shrink; on a GPU of its own the call is
 * slower that way. Results differ only within rounding (other split boundaries); each plan is
 * deterministic. */
#define HISPARSE_ATTN_BESIDE_FETCH 2
/* hisparse_attn_desc_t.flags, a scheduling hint for latent attention: the call carries an
 * exact-prefetch replay (hisparse_sparse_decode_prefetch, _part) whose host-link transfer takes
 * longer than the attention itself, so the launch lasts as long as the replay and the merge that
 * follows it sits on the decode chain (Section 3.5). With one token group per workgroup (few
 * workgroup columns, e.g. one request of 128 heads) the plan then takes splits of at least 4
 * chunks instead of 2: half the attention workgroups, which stay hidden behind the replay and
 * leave it more CUs, and half the split partials for the merge to read. Set it on the carrying
 * call and on its hisparse_attention_merge (or _merge_prefetch). Results differ only within
 * rounding (other split boundaries); each plan is deterministic. */
#define HISPARSE_ATTN_CARRIES_REPLAY 4

/* Human-readable name of a status code (static storage). */
const char* hisparse_status_string(hisparse_status_t status);

/* [pure host] Check a cache descriptor without touching any device. */
hisparse_status_t hisparse_validate_desc(const hisparse_cache_desc_t* desc);

/* [pure host] Check an attention descriptor against a cache descriptor's record layout. */
hisparse_status_t hisparse_validate_attn(int32_t record_bytes, int32_t top_k,
                                         const hisparse_attn_desc_t* attn);

/* [sync] Create a cache on HIP device `device`. Allocates, and owns until destroy:
 *   - per layer, a pinned mapped host pool [units][L][R] (the authoritative full KV,
 *     Section 3.2 "host KV pool"), uninitialised -- the caller stages prefill KV into it
 *     (hisparse_host_pool) before resolving;
 *   - per layer, the GPU cache [units][B][R] in HBM;
 *   - per anchor layer, the page table [units][L] int32 (-1 = host-only), slot map [units][B]
 *     int32 (-1 = empty), LRU timestamps [units][B] uint32, recency index [units][B], step clock
 *     [units] and miss plan [units][k] -- all initialised to the cold state.
 * On failure nothing stays allocated and *out is NULL. */
hisparse_status_t hisparse_cache_create(const hisparse_cache_desc_t* desc, int32_t device,
                                        hisparse_cache_t* out);

/* [sync] Release everything the handle owns. NULL is accepted. */
hisparse_status_t hisparse_cache_destroy(hisparse_cache_t cache);

/* Host address and size of layer `layer`'s pinned host pool, laid out [units][L][R]: record r
 * of unit u starts at host + (u * L + r) * R. The caller may write it whenever no GPU work
 * that reads it is in flight. */
hisparse_status_t hisparse_host_pool(hisparse_cache_t cache, int32_t layer, void** host,
                                     size_t* bytes);

/* Device address and size of layer `layer`'s GPU cache, laid out [units][B][R]. */
hisparse_status_t hisparse_layer_cache(hisparse_cache_t cache, int32_t layer, void** device,
                                       size_t* bytes);

/* [async] Return every anchor layer's units to the cold state (all slots empty, clocks 0). */
hisparse_status_t hisparse_reset(hisparse_cache_t cache, void* stream);

/* ---- Request lifecycle (Section 3.3 (1) prefill and staging, (2) admission) ----
 * A cache reserves every unit's slot caches and tables for all its layers when it is created
 * (num_layers * B * R bytes of slots per unit, the per-request reservation Section 3.3 (2)
 * sizes by B rather than by context length), so admitting a request allocates nothing: it takes
 * one of num_requests request slots, whose units are
 * [request * units_per_request, (request + 1) * units_per_request). */

/* Take a free request slot, lowest index first (host bookkeeping; no GPU work, and the kernels
 * do not consult it). All slots are free after creation. Returns HISPARSE_ERR_FULL, leaving
 * *request = -1, when every slot is taken. */
hisparse_status_t hisparse_request_acquire(hisparse_cache_t cache, int32_t* request);

/* [async] Give a request slot back: its units go back to the cold state in every anchor layer
 * (hisparse_reset_units on `stream`) and the slot is free for the next acquire at once, so
 * work for the next request on those units must be ordered after this call by `stream`.
 * Returns INVALID_ARG for a slot that is out of range or not taken. */
hisparse_status_t hisparse_request_release(hisparse_cache_t cache, int32_t request,
                                           void* stream);

/* [async] Cold state for units [first_unit, first_unit + num_units) of every anchor layer, as
 * after creation: page-table rows cleared, slots empty, stamps and clocks 0, recency index in
 * slot order, miss plans empty. Other units, the GPU caches' bytes and the host pools are
 * untouched. 1 <= num_units, first_unit + num_units <= units. */
hisparse_status_t hisparse_reset_units(hisparse_cache_t cache, int32_t first_unit,
                                       int32_t num_units, void* stream);

/* [async] Prefill staging (Section 3.3 (1)): copy records [first_record, first_record +
 * num_records) of units [first_unit, first_unit + num_units) of layers [first_layer,
 * first_layer + num_layers) from device memory into the host pools with the copy engines
 * (device-to-host hipMemcpyAsync, one per layer when num_records = L or num_units = 1, else one
 * per unit and layer).
 *   d_src  device; layer first_layer + j at d_src + j * src_layer_stride, laid out
 *          [num_units][num_records][R] (not modified).
 *   src_layer_stride  bytes, >= num_units * num_records * R; ignored when num_layers = 1.
 * The records may be resolved once this work has completed (the staging acknowledgement: an
 * event the caller records on `stream` after the call). The staged range must not be read by
 * fetches in flight. Capturable in a HIP graph. */
hisparse_status_t hisparse_stage(hisparse_cache_t cache, int32_t first_layer, int32_t num_layers,
                                 int32_t first_unit, int32_t num_units, int64_t first_record,
                                 int64_t num_records, const void* d_src,
                                 int64_t src_layer_stride, void* stream);

/* [async] Resolve one step of an anchor layer (Section 3.4 phases 1-5).
 *   d_sel    int32 [units][k]: selected positions per unit, in the indexer's order.
 *   d_slots  int32 [units][k]: out; d_slots[u][i] is the slot of unit u now holding record
 *            d_sel[u][i] (Section 3.3 (3): aligned with the selection's order); -1 for padding.
 *   d_counts int32 [units][2]: out, {hits, misses} per unit; may be NULL.
 * Replacement is LRU among the slots the step does not reference, with this step's hits
 * promoted above its newly fetched misses (Section 3.2 "Replacement policy"). Ties are
 * canonical: misses of step t are stamped 2t-1 and hits 2t (t = the unit's valid steps so
 * far + 1); victims are taken in ascending (timestamp, slot) order, empty slots first, and
 * the i-th miss in ascending position order takes the i-th victim. Misses are fetched from
 * this layer's host pool (unless fetch = HISPARSE_FETCH_NONE), and the miss plan is kept for
 * hisparse_prefetch_layer. Returns INVALID_ARG for a shared (non-anchor) layer. */
hisparse_status_t hisparse_resolve(hisparse_cache_t cache, int32_t layer, const int32_t* d_sel,
                                   int32_t* d_slots, int32_t* d_counts, void* stream);

/* [async] The two halves of hisparse_resolve, for callers that schedule or time them apart
 * (the paper's breakdown of a resolve into metadata phases and IO, Section 4.4):
 * hisparse_resolve_tables runs phases 1-3 and 5 -- every output of hisparse_resolve and the
 * miss plan, but no record is copied; hisparse_fetch then runs phase 4, copying the records of
 * the anchor layer's latest miss plan from its host pool into its GPU cache (a no-op under
 * HISPARSE_FETCH_NONE). hisparse_resolve == hisparse_resolve_tables + hisparse_fetch. */
hisparse_status_t hisparse_resolve_tables(hisparse_cache_t cache, int32_t layer,
                                          const int32_t* d_sel, int32_t* d_slots,
                                          int32_t* d_counts, void* stream);
hisparse_status_t hisparse_fetch(hisparse_cache_t cache, int32_t layer, void* stream);

/* [async] Phase 4 for entries [m * part_begin / 256, m * part_end / 256) of each unit's plan
 * of m entries only, 0 <= part_begin <= part_end <= 256: calls over adjacent ranges together
 * equal hisparse_fetch. A caller that hands the host link from one stream to another can let
 * the next stream's transfer start after the first part (an event recorded between the calls)
 * while the rest of this one still runs. */
hisparse_status_t hisparse_fetch_part(hisparse_cache_t cache, int32_t layer, int32_t part_begin,
                                      int32_t part_end, void* stream);

/* [async] hisparse_fetch (Section 3.4 Phase 4) taking turns on the host link with fetches
 * issued on other streams, ordered on the device instead of by stream events. The paper
 * overlaps the fetch with other work so that IO stays off the critical path (Section 3.5);
 * with several independent batches of units, each with its own stream, one batch's fetch
 * overlaps another's attention best when the fetches use the link one after another.
 *   d_turns int32 [2 * n_turns] (n_turns >= 1), device memory owned by the caller, zeroed with
 *     hisparse_link_turns_reset before the first launch of a sequence of turns; turn i is
 *     the pair d_turns[2i], d_turns[2i + 1]. Each turn is signalled by one launch and waited
 *     for by at most one.
 *   wait_turn: -1, or the turn whose signal this launch waits for before its first host
 *     read. The launch's waves are resident while they wait, polling d_turns.
 *   signal_turn: -1, or the turn this launch signals once signal_share / 256 (1..256) of its
 *     workgroups have finished their copies (256: all of them, the link free).
 * The copies and results equal hisparse_fetch's whatever the order of the launches: a turn
 * orders only the use of the link, never data. A wait ends by itself after about 4 ms once
 * the signalling launch has started, or after about 50 us if it has not (not yet issued, or
 * queued behind this launch), so a turn that cannot be signalled in time (reset missing, its
 * launch on a stream that waits for this one, launches serialised by a tool) costs time, not
 * correctness. For a sequence issued on streams that may run concurrently.
 * HISPARSE_ERR_UNSUPPORTED unless the cache fetches zero-copy (the host-issued paths and
 * HISPARSE_FETCH_NONE launch no kernel); INVALID_ARG for a shared layer, a null d_turns,
 * n_turns < 1, indices outside [-1, n_turns), wait_turn == signal_turn, or a share outside
 * 1..256. */
hisparse_status_t hisparse_fetch_turn(hisparse_cache_t cache, int32_t layer, int32_t* d_turns,
                                      int32_t n_turns, int32_t wait_turn, int32_t signal_turn,
                                      int32_t signal_share, void* stream);

/* [async] Zero n_turns (1..2^24) link turns, d_turns[0 .. 2 * n_turns), with a fill kernel on
 * `stream` (capturable; no memset node), launched on the calling thread's current HIP device,
 * which must hold d_turns and `stream`. See hisparse_fetch_turn. */
hisparse_status_t hisparse_link_turns_reset(int32_t* d_turns, int32_t n_turns, void* stream);

/* [async] Phase 4 for units [unit_begin, unit_begin + unit_count) of an anchor layer only
 * (Section 3.4; units are independent caches). Calls over disjoint ranges together equal
 * hisparse_fetch, so a caller can pipeline a layer's fetch with the attention of the units
 * already fetched. HISPARSE_ERR_INVALID_ARG for a range outside [0, units). */
hisparse_status_t hisparse_fetch_units(hisparse_cache_t cache, int32_t layer,
                                       int32_t unit_begin, int32_t unit_count, void* stream);

/* [async] Phase 4 of an anchor layer and the exact-prefetch replay of the same miss plan into
 * its next num_layers - 1 shared layers (Section 3.5), in one launch: equal to hisparse_fetch
 * followed by hisparse_prefetch_layer for each of those layers, for a caller with nothing to
 * overlap the replays with. HISPARSE_ERR_INVALID_ARG unless 1 <= num_layers <= share_group and
 * the layers exist. */
hisparse_status_t hisparse_fetch_group(hisparse_cache_t cache, int32_t anchor_layer,
                                       int32_t num_layers, void* stream);

/* [async] Exact prefetch (Section 3.5): replay the miss plan recorded by the latest resolve of
 * `anchor_layer` into the cache of `shared_layer` (anchor < shared < anchor + share_group),
 * copying each planned record from shared_layer's own host pool into the same slot. After the
 * replay, shared_layer's cache holds its records for the anchor's selection in the anchor's
 * slots, so its attention reads through the anchor's d_slots. The caller orders it after that
 * resolve (e.g. an event) and before the shared layer's attention, and must not start the
 * anchor's next resolve before the replay has completed. */
hisparse_status_t hisparse_prefetch_layer(hisparse_cache_t cache, int32_t anchor_layer,
                                          int32_t shared_layer, void* stream);

/* [async] hisparse_prefetch_layer for the num_layers consecutive shared layers first_shared ..
 * first_shared + num_layers - 1 of `anchor_layer`'s group, in one launch (Section 3.5): the
 * side-stream form of the replay, started as soon as the anchor's resolve has recorded its
 * plan, so that it shares the host link with the anchor's own fetch and runs under the anchor
 * layer's attention. Same ordering rules as hisparse_prefetch_layer. HISPARSE_ERR_INVALID_ARG
 * unless anchor < first_shared and first_shared + num_layers <= min(anchor + share_group,
 * num_layers), num_layers >= 1. */
hisparse_status_t hisparse_prefetch_layers(hisparse_cache_t cache, int32_t anchor_layer,
                                           int32_t first_shared, int32_t num_layers,
                                           void* stream);

/* [async] Speculative cross-layer prefetch for models whose layers do not share selections
 * (Section 3.5, the speculative alternative to exact prefetch): anchor layer `layer` takes a
 * hint, typically the previous layer's selection of the same step, as one access event of its
 * canonical LRU, exactly as hisparse_resolve would take it as a selection: the layer's clock
 * advances, hinted records already resident are refreshed, the others are fetched into its
 * least-recent slots. Its own resolve later in the step then finds them resident. No slot
 * vector is written.
 *   d_hint   int32 [units][k], positions in [0, L) or -1 for padding (invalid entries latch
 *            HISPARSE_ERR_BAD_SELECTION as in hisparse_resolve).
 *   d_counts int32 [units][2]: out, {already resident, fetched} per unit; may be NULL.
 * A wrong hint costs transfers and evictions, never correctness: the layer's resolve still
 * makes every selected record resident. The hint replaces the layer's miss plan, so replays
 * into shared layers (hisparse_prefetch_layer) must follow the layer's own resolve. */
hisparse_status_t hisparse_speculate(hisparse_cache_t cache, int32_t layer,
                                     const int32_t* d_hint, int32_t* d_counts, void* stream);

/* [async] Write-through of generated records (Section 3.3 (4)): each unit's newly generated
 * record enters the GPU caches of layers [first_layer, first_layer + num_layers) and is written
 * through to those layers' host pools, in one launch. The range covers whole share groups:
 * first_layer is an anchor and the range ends at a group boundary or at the last layer.
 *   d_pos     int32 [units]: the new record's position per unit (< 0: nothing for that unit;
 *             >= num_records: HISPARSE_ERR_BAD_SELECTION latched, state unchanged).
 *   d_records bf16 records [num_layers][units][R].
 *   d_slots   int32 [groups in the range][units], out: the slot the position now occupies in
 *             each group (-1: none).
 * Each group's anchor admits the position as a one-entry resolve event: the unit's clock
 * advances by one; a resident position is refreshed in place, otherwise the least-recent slot
 * by (timestamp, slot) takes it with the event's miss stamp, exactly as the canonical LRU does
 * for a selection {pos}. Each layer's record is then stored into that slot of the layer's cache
 * and into position pos of the layer's host pool, by the GPU over the mapped pool, so any later
 * fetch of pos on a stream ordered after this call reads it. Order the call after every
 * attention that reads the slots of the groups' current step (an admission may evict one of
 * them) and before those anchors' next resolve; the resolves' miss plans are left intact.
 * HISPARSE_FETCH_NONE updates the tables only. */
hisparse_status_t hisparse_append(hisparse_cache_t cache, int32_t first_layer,
                                  int32_t num_layers, const int32_t* d_pos,
                                  const void* d_records, int32_t* d_slots, void* stream);

/* Bytes of device workspace hisparse_sparse_decode(_pool) needs for `units` units of top_k
 * records each; 0 if the descriptor is invalid. */
size_t hisparse_decode_workspace_bytes(int32_t units, int32_t top_k, int32_t record_bytes,
                                       const hisparse_attn_desc_t* attn);

/* [async] Sparse decode attention of one layer over its GPU cache (the consumer of Section 3.4
 * Phase 5's slot vector).
 *   d_q     bf16 [units][q_heads][d_qk] query.
 *   d_slots int32 [units][k]: slots from hisparse_resolve (the anchor's, for a shared layer);
 *           -1 entries are skipped.
 *   d_out   float32 [units][q_heads][d_v]: out_h = sum_j softmax_j(scale * q_h . key_j) value_j
 *           over the tokens of the selected records. A unit with no valid record gets zeros.
 *   d_workspace / workspace_bytes: caller-owned scratch of at least
 *           hisparse_decode_workspace_bytes(units, k, R, attn) bytes.
 * The reduction order depends only on the position of a record in the slot vector, never on
 * the slot value, so the result is bit-identical to hisparse_sparse_decode_pool over any other
 * placement of the same records. */
hisparse_status_t hisparse_sparse_decode(hisparse_cache_t cache, int32_t layer, const void* d_q,
                                         const int32_t* d_slots, float* d_out,
                                         const hisparse_attn_desc_t* attn, void* d_workspace,
                                         size_t workspace_bytes, void* stream);

/* [async] The merge of an attention call made with HISPARSE_ATTN_DEFER_MERGE: combines the
 * per-split partial results in d_workspace into d_out (float32 [units][q_heads][d_v]), in
 * the fixed split order, so deferred call + merge == the same call without the flag, bit for
 * bit. units, top_k, record_bytes and attn (HISPARSE_ATTN_DEFER_MERGE aside) must be those of
 * the deferred call,
 * whose `units` is the cache's units times the layer count for hisparse_sparse_decode_layers;
 * the workspace must not be reused in between. */
hisparse_status_t hisparse_attention_merge(int32_t units, int32_t top_k, int32_t record_bytes,
                                           const hisparse_attn_desc_t* attn, float* d_out,
                                           const void* d_workspace, size_t workspace_bytes,
                                           void* stream);

/* Bytes of device scratch each GPU holds for hisparse_sparse_decode_noalloc (64 MiB). */
#define HISPARSE_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* [async] hisparse_sparse_decode without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the split partial results go to a scratch array of HISPARSE_NOALLOC_SCRATCH_BYTES that the
 * library holds on each GPU it runs on until the process ends, and the call allocates nothing.
 * Same arguments, output and bits as hisparse_sparse_decode with a workspace.
 *   - HISPARSE_ERR_UNSUPPORTED if the call needs more scratch than that
 *     (hisparse_decode_workspace_bytes(units, k, R, attn) > HISPARSE_NOALLOC_SCRATCH_BYTES);
 *   - HISPARSE_ERR_INVALID_ARG with HISPARSE_ATTN_DEFER_MERGE (the partials have no owner).
 * Every call on one GPU shares that GPU's scratch, from any handle: calls that may overlap on
 * one GPU (other streams, other host threads) race and must be ordered by the caller. */
hisparse_status_t hisparse_sparse_decode_noalloc(hisparse_cache_t cache, int32_t layer,
                                                 const void* d_q, const int32_t* d_slots,
                                                 float* d_out, const hisparse_attn_desc_t* attn,
                                                 void* stream);

/* [async] hisparse_sparse_decode of `layer` and, in the same launch, the exact-prefetch replay
 * of `anchor_layer`'s latest plan into shared layers [first_shared, first_shared + num_shared)
 * (Section 3.5): equal to hisparse_prefetch_layers followed by hisparse_sparse_decode, but the
 * replay runs in extra workgroups beside the attention, so the next layers' misses cross the
 * host link while this layer attends, on one stream. Ordering rules of
 * hisparse_prefetch_layer apply to the replay. With HISPARSE_FETCH_SDMA the replay is issued
 * on its own first (host-synchronising); with HISPARSE_FETCH_NONE nothing is copied.
 * HISPARSE_ERR_INVALID_ARG for a replay range hisparse_prefetch_layers would refuse, for
 * num_shared > 8, or if `layer` is one of the replay's targets. */
hisparse_status_t hisparse_sparse_decode_prefetch(hisparse_cache_t cache, int32_t layer,
                                                  const void* d_q, const int32_t* d_slots,
                                                  float* d_out, const hisparse_attn_desc_t* attn,
                                                  void* d_workspace, size_t workspace_bytes,
                                                  int32_t anchor_layer, int32_t first_shared,
                                                  int32_t num_shared, void* stream);

/* [async] hisparse_sparse_decode_prefetch carrying only part of the replay: entries
 * [m * part_begin / 256, m * part_end / 256) of each unit's plan of m entries, 0 <= part_begin
 * <= part_end <= 256 (0, 256: all of it, i.e. hisparse_sparse_decode_prefetch). Calls with
 * adjacent ranges, e.g. one carried by hisparse_attention_merge_prefetch and the rest by this
 * call, copy every planned record exactly once. Same ordering rules and errors. */
hisparse_status_t hisparse_sparse_decode_prefetch_part(
    hisparse_cache_t cache, int32_t layer, const void* d_q, const int32_t* d_slots,
    float* d_out, const hisparse_attn_desc_t* attn, void* d_workspace, size_t workspace_bytes,
    int32_t anchor_layer, int32_t first_shared, int32_t num_shared, int32_t part_begin,
    int32_t part_end, void* stream);

/* [async] hisparse_attention_merge of a deferred attention call made on `cache` (its units, top
 * k and record size; attn as in that call) whose launch also carries part of an exact-prefetch
 * replay (Section 3.5): entries [m * part_begin / 256, m * part_end / 256) of each unit's plan of
 * `anchor_layer`, into shared layers [first_shared, first_shared + num_shared), in extra
 * workgroups beside the merge. For a decode loop whose every attention call carries the replay
 * into a later shared layer, the merges would otherwise leave the host link idle; starting the
 * next-but-one layer's replay in them keeps it busy, and the attention call that follows carries
 * the rest (hisparse_sparse_decode_prefetch_part). Ordering rules of hisparse_prefetch_layer
 * apply to the replay. HISPARSE_ERR_INVALID_ARG for a replay range
 * hisparse_sparse_decode_prefetch_part would refuse. */
hisparse_status_t hisparse_attention_merge_prefetch(hisparse_cache_t cache,
                                                    const hisparse_attn_desc_t* attn,
                                                    float* d_out, const void* d_workspace,
                                                    size_t workspace_bytes, int32_t anchor_layer,
                                                    int32_t first_shared, int32_t num_shared,
                                                    int32_t part_begin, int32_t part_end,
                                                    void* stream);

/* [async] Sparse decode attention of layers [first_layer, first_layer + num_layers) of one
 * share group in a single launch (Section 3.5: the shared layers read their records through
 * the anchor's slots; batching them is this library's scheduling choice, the result per layer
 * is the same attention as hisparse_sparse_decode up to the split boundaries).
 *   d_q     bf16 [num_layers][units][q_heads][d_qk].
 *   d_slots int32 [units][k]: the anchor's slot vector, read by every layer.
 *   d_out   float32 [num_layers][units][q_heads][d_v].
 *   d_workspace / workspace_bytes: at least
 *           hisparse_decode_workspace_bytes(num_layers * units, k, R, attn) bytes.
 * HISPARSE_ERR_INVALID_ARG if the layers span two share groups. */
hisparse_status_t hisparse_sparse_decode_layers(hisparse_cache_t cache, int32_t first_layer,
                                                int32_t num_layers, const void* d_q,
                                                const int32_t* d_slots, float* d_out,
                                                const hisparse_attn_desc_t* attn,
                                                void* d_workspace, size_t workspace_bytes,
                                                void* stream);

/* [async] The same attention over an explicit device pool [units][records_per_unit][R], with
 * d_idx int32 [units][k] record indices into each unit's part of the pool (-1 = skip). Used for
 * a fully resident KV (indices = positions), or any other placement. One unit's part of the
 * pool, records_per_unit * R bytes, must stay below 2 GiB (HISPARSE_ERR_UNSUPPORTED otherwise;
 * the same holds for B * R of a cache). */
hisparse_status_t hisparse_sparse_decode_pool(const void* d_pool, int64_t records_per_unit,
                                              int32_t record_bytes, int32_t units, int32_t top_k,
                                              const void* d_q, const int32_t* d_idx, float* d_out,
                                              const hisparse_attn_desc_t* attn,
                                              void* d_workspace, size_t workspace_bytes,
                                              void* stream);

/* [sync] Copy an anchor layer's resolve state into host buffers (any may be NULL):
 * slot_pos int32 [units][B], slot_ts uint32 [units][B], page_table int32 [units][L],
 * order int32 [units][B] (slots by ascending (timestamp, slot)), clock uint32 [units]. */
hisparse_status_t hisparse_read_state(hisparse_cache_t cache, int32_t layer, int32_t* slot_pos,
                                      uint32_t* slot_ts, int32_t* page_table, int32_t* order,
                                      uint32_t* clock);

/* [sync] Copy an anchor layer's latest miss plan into host buffers (either may be NULL):
 * plan int32 [units][k][2] = (position, slot) for the first count[u] entries, in ascending
 * position order; count int32 [units]. */
hisparse_status_t hisparse_read_plan(hisparse_cache_t cache, int32_t layer, int32_t* plan,
                                     int32_t* count);

/* [sync] Return HISPARSE_ERR_BAD_SELECTION if a device-side selection error was latched since
 * the last check (info, if not NULL, receives {layer, unit, number of failing unit-steps}),
 * clearing the latch; otherwise HISPARSE_OK. */
hisparse_status_t hisparse_check_errors(hisparse_cache_t cache, int32_t* info);

/* Stamps per unit of the resolve kernel's phase timing (see hisparse_debug_resolve_phases). */
#define HISPARSE_RESOLVE_PHASE_SLOTS 16
/* The first units whose resolve workgroups record phase stamps. */
#define HISPARSE_RESOLVE_PHASE_UNITS 64

/* [sync] Diagnostic, Section 4.4's breakdown of the resolve into its phases: in a library built
 * with HISPARSE_PHASE_STAMPS (`python -m paper_2608_07009_amd.build --phase-stamps`, which
 * writes lib/libhisparse_phase_stamps.so), the resolve kernel stores the device's constant-rate
 * wall clock at its phase boundaries, for units below HISPARSE_RESOLVE_PHASE_UNITS, overwriting
 * the previous launch's stamps. This call waits for the current device and copies the stamps of
 * the first min(max_units, HISPARSE_RESOLVE_PHASE_UNITS) units into host_stamps (uint64
 * [units][HISPARSE_RESOLVE_PHASE_SLOTS], caller-owned): slot 0 kernel start, 1 selection staged
 * and probed (phase 1), 2 misses bucketed, 3 bucket starts scanned, 4 misses in position order
 * (phase 2), 5 victims chosen (phase 3a), 6 recency index and hit stamps written (phase 3b),
 * 7 tables, plan and slots updated (phase 5), 8 kernel end; slots 9.. are unused. A unit whose
 * selection was invalid stops after slot 4. ticks_per_s (if not NULL) receives the clock's rate.
 * Launches on several streams at once overwrite each other's stamps. In a normal build it
 * returns HISPARSE_ERR_UNSUPPORTED and touches nothing. */
hisparse_status_t hisparse_debug_resolve_phases(uint64_t* host_stamps, int32_t max_units,
                                                int64_t* ticks_per_s);

#ifdef __cplusplus
}
#endif

#endif /* HISPARSE_H */
