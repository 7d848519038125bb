// Internal declarations shared by the HiSparse HIP library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "gather_pool.h"
#include "hisparse.h"

namespace hisparse {

constexpr int kMaxTopK = 4096;
constexpr int kMaxCapacity = 16384;
constexpr int kMaxRecordBytes = 1 << 20;
// Sparse decode attention: tokens of one workgroup split (validity bitmask in LDS), and the most
// split partial results the latent-attention merge takes per (unit, head) (weights in LDS). A
// latent-attention call therefore covers at most kMlaMaxParts * kMaxSplitTokens tokens per unit.
constexpr int kMaxSplitTokens = 8192;
constexpr int kMlaMaxParts = 128;

// Error word layout: [0] first error code, [1] layer, [2] unit, [3] failing unit-steps.
constexpr int kErrWords = 4;

struct ResolveArgs {
  const int32_t* sel;   // [units][k]
  int32_t* pt;          // [units][L]
  int32_t* slot_pos;    // [units][B]
  uint32_t* slot_ts;    // [units][B]
  int32_t* order;       // [units][B], slots by ascending (ts, slot)
  uint32_t* clock;      // [units]
  int32_t* slots_out;   // [units][k]
  int32_t* counts_out;  // [units][2]
  int2* plan;           // [units][k] (position, slot)
  int32_t* plan_count;  // [units]
  int32_t* err;         // [kErrWords]
  int64_t L;
  int32_t B, k, layer, units;
};

constexpr int kMaxFetchLayers = 8;  // layers one fetch launch serves (grid z)

struct FetchArgs {
  const int2* plan;         // [units][k]
  const int32_t* plan_count;  // [units]
  const uint8_t* host[kMaxFetchLayers];  // per target layer: device-visible host pool [units][L][R]
  uint8_t* cache;           // first target layer's GPU cache [units][B][R]
  int64_t cache_stride;     // bytes from one target layer's cache to the next
  int64_t L;
  int32_t B, k, R, units, n_layers;
  // each unit's plan entries [m * part_lo / 256, m * part_hi / 256) of its m (0, 256: all), so
  // that launches with adjacent ranges split one copy exactly
  int32_t part_lo, part_hi;
};

// Device tables the write-through kernel indexes: per anchor its resolve state, per layer its
// GPU cache and the device-visible address of its host pool.
struct AnchorState {
  int32_t* pt;          // [units][L]
  int32_t* slot_pos;    // [units][B]
  uint32_t* slot_ts;    // [units][B]
  int32_t* order;       // [units][B]
  uint32_t* clock;      // [units]
};
struct LayerIO {
  uint8_t* cache;       // [units][B][R]
  uint8_t* host;        // [units][L][R]
};

// Write-through of generated records for layers [first, first + n_layers), whole share groups:
// each group's anchor admits the unit's new position (the canonical LRU on the one-entry
// selection {pos}) and the group's layers receive their records in that slot and at pos in
// their host pools.
struct AdmitArgs {
  const int32_t* pos;          // [units] the new position (< 0: none this event)
  const AnchorState* states;   // [anchors]
  const LayerIO* layers;       // [num_layers]
  const uint8_t* records;      // [n_layers][units][R]
  int32_t* slots_out;          // [groups in range][units]
  int32_t* err;                // [kErrWords]
  int64_t L;
  int32_t B, R, units, G, first, n_layers, write;  // write = 0: tables only
};

struct StateArgs {
  int32_t* pt;
  int32_t* slot_pos;
  uint32_t* slot_ts;
  int32_t* order;
  uint32_t* clock;
  int32_t* plan_count;
  int64_t L;
  int32_t B, units;
};

// Staged fetch: records packed per unit in a device staging buffer, each unit's run starting at
// entry prefix[u] (prefix: [units + 1] int32 at the buffer's start, records from rec_offset).
struct ScatterArgs {
  const uint8_t* stage;        // device staging buffer
  const int2* plan;            // [units][k] (position, slot)
  const int32_t* plan_count;   // [units]
  uint8_t* cache;              // [units][B][R]
  int64_t rec_offset;          // bytes before the first record
  int32_t B, k, R, units;
  int32_t part_lo;             // unit u's packed run is its plan entries from m * part_lo / 256
};

hipError_t launch_resolve(const ResolveArgs& a, hipStream_t stream);
// Phase stamps of the last resolve launch (phase-timing builds only; else hipErrorNotSupported).
constexpr int kPhaseStamps = HISPARSE_RESOLVE_PHASE_SLOTS;
constexpr int kPhaseStampUnits = HISPARSE_RESOLVE_PHASE_UNITS;
hipError_t read_resolve_phase_stamps(uint64_t* host, int32_t units);
hipError_t launch_scatter(const ScatterArgs& a, hipStream_t stream);
hipError_t launch_fetch(const FetchArgs& a, int transfer_block_bytes, int workgroups,
                        hipStream_t stream);
hipError_t launch_reset_state(const StateArgs& a, hipStream_t stream);
hipError_t launch_admit(const AdmitArgs& a, int32_t n_groups, hipStream_t stream);
size_t resolve_lds_bytes(int32_t k, int32_t B);
int resolve_threads(int32_t B);

// Attention over records addressed by idx[unit][k] (entries outside [0, records_per_unit) are skipped) into pool[unit][records_per_unit][R].
struct AttnPlan {
  int32_t hw, tw, hb;        // head waves, token waves, head blocks
  int32_t tg;                // latent attention: token groups merged within a workgroup
  int32_t n_tok;             // tokens per unit = k * tokens_per_record
  int32_t split_tokens;      // tokens per workgroup split (multiple of 32 * tw)
  int32_t n_wg_splits;       // workgroup splits per unit
  int32_t n_parts;           // partial results per (unit, head) = n_wg_splits * tw
  size_t workspace_bytes;
};
hisparse_status_t plan_attention(int32_t units, int32_t top_k, int32_t record_bytes,
                                 const hisparse_attn_desc_t* attn, AttnPlan* plan);
// The merge of the per-split partials in `workspace` into out (skipped by launch_attention
// when attn.flags has HISPARSE_ATTN_DEFER_MERGE).
hipError_t launch_merge(const AttnPlan& p, const hisparse_attn_desc_t& attn, int32_t units,
                        float* out, const void* workspace, hipStream_t stream,
                        const FetchArgs* prefetch = nullptr, int32_t prefetch_threads = 0,
                        int32_t prefetch_block_bytes = 16);
hipError_t launch_attention(const AttnPlan& p, const hisparse_attn_desc_t& attn,
                            const uint8_t* pool, int64_t records_per_unit, int32_t record_bytes,
                            int32_t units, int32_t top_k, const uint16_t* q, const int32_t* idx,
                            float* out, void* workspace, hipStream_t stream,
                            int32_t idx_units = 0, const FetchArgs* prefetch = nullptr,
                            int32_t prefetch_threads = 0, int32_t prefetch_block_bytes = 16);

}  // namespace hisparse

struct hisparse_cache {
  hisparse_cache_desc_t desc;
  int device = 0;
  int32_t units = 0;
  int32_t n_anchors = 0;
  size_t host_layer_bytes = 0;
  size_t cache_layer_bytes = 0;
  std::vector<void*> host;       // per layer, host address of the pinned pool
  std::vector<void*> host_dev;   // per layer, device-visible address of the same pool
  uint8_t* cache_all = nullptr;  // GPU caches of all layers, one allocation [layer][unit][B][R]
  std::vector<uint8_t*> cache;   // per layer, GPU cache (into cache_all)
  struct Anchor {
    int32_t* pt = nullptr;
    int32_t* slot_pos = nullptr;
    uint32_t* slot_ts = nullptr;
    int32_t* order = nullptr;
    uint32_t* clock = nullptr;
    int2* plan = nullptr;
    int32_t* plan_count = nullptr;
    int32_t* counts = nullptr;   // used when the caller passes no counts buffer
  };
  hisparse::AnchorState* d_states = nullptr;  // device copies of every anchor's state pointers
  hisparse::LayerIO* d_layers = nullptr;      // and of every layer's cache / host pool address
  std::vector<Anchor> anchors;   // per anchor layer (layer / share_group)
  std::vector<uint8_t> request_taken;  // request slots handed out by hisparse_request_acquire
  int32_t* err = nullptr;        // device error word
  // HISPARSE_FETCH_SDMA / _STAGED: pinned readback of a plan and the host-side copy lists
  int32_t* h_plan_count = nullptr;
  int2* h_plan = nullptr;
  std::vector<void*> dma_dst, dma_src;
  std::vector<size_t> dma_size;
  // HISPARSE_FETCH_STAGED: pinned and device staging buffers ([units + 1] prefix, then up to
  // units * top_k records) and the host threads that gather into the pinned one
  uint8_t* stage_host = nullptr;
  uint8_t* stage_dev = nullptr;
  size_t stage_bytes = 0;
  hipEvent_t stage_done = nullptr;  // recorded after the last staged fetch's scatter
  hisparse::GatherPool* gather = nullptr;
};
