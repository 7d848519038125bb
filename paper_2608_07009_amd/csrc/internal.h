// Internal declarations shared by the HiSparse HIP library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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
// Host-link turns between fetch launches on different streams (hisparse_fetch_turn): turn i
// is the word pair turns[2i] (finished workgroups of the launch that signals it) and
// turns[2i + 1] (1 once that launch has started, 2 once the launch that waits for it may
// start reading).
struct LinkTurn {
  int32_t* turns;  // null: no turn taking
  int32_t wait;    // turn to wait for before the first host read (-1: none)
  int32_t signal;  // turn to signal (-1: none)
  int32_t share;   // 1..256: the 256ths of this launch's workgroups that finish before it does
};
hipError_t launch_fetch(const FetchArgs& a, int transfer_block_bytes, int workgroups,
                        hipStream_t stream, const LinkTurn* turn = nullptr);
hipError_t launch_turns_reset(int32_t* turns, int32_t n_turns, hipStream_t stream);
hipError_t launch_reset_state(const StateArgs& a, hipStream_t stream);
hipError_t launch_admit(const AdmitArgs& a, int32_t n_groups, hipStream_t stream);
size_t resolve_lds_bytes(int32_t k, int32_t B);
int resolve_threads(int32_t B);

// Attention over records addressed by idx[unit][k] (entries outside [0, records_per_unit) are skipped) into pool[unit][records_per_unit][R].
struct AttnPlan {
  int32_t hw, tw, hb;        // head waves, token waves, head blocks
  int32_t tg;                // latent attention: token groups merged within a workgroup
  bool paced;                // latent attention: the query loaded after the first chunks
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
