// The cache handle behind hisparse_cache_t: host-side state of the library's entry points
// (included by the C ABI's translation unit only; the kernels never see it).
#pragma once

#include <vector>

#include "gather_pool.h"
#include "internal.h"

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
