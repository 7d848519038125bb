// C ABI of the HiSparse library: descriptor validation, allocation of the host pool, GPU
// cache and resolve state, and the enqueueing entry points (declared in include/hisparse.h).
#include <dlfcn.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>

#include "handle.h"

using hisparse::kMaxCapacity;
using hisparse::kMaxRecordBytes;
using hisparse::kMaxTopK;

// Dynamic LDS the resolve kernel may take: a gfx950 workgroup's 160 KiB less 256 bytes for the
// kernel's own scan scratch.
constexpr size_t kMaxResolveLds = 160 * 1024 - 256;

namespace {

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// hipMemcpyBatchAsync exists only in newer HIP runtimes; the process may run an older one
// (whichever libamdhip64 was loaded first), so it is looked up at run time.
typedef hipError_t (*batch_copy_fn)(void**, void**, size_t*, size_t, hipMemcpyAttributes*,
                                    size_t*, size_t, size_t*, hipStream_t);
batch_copy_fn batch_copy() {
  static batch_copy_fn fn =
      reinterpret_cast<batch_copy_fn>(dlsym(RTLD_DEFAULT, "hipMemcpyBatchAsync"));
  return fn;
}

bool is_anchor(const hisparse_cache* c, int32_t layer) {
  return layer >= 0 && layer < c->desc.num_layers && layer % c->desc.share_group == 0;
}

int transfer_block(const hisparse_cache_desc_t& d) {
  return d.transfer_block_bytes == 0 ? 16 : d.transfer_block_bytes;
}

// The default fetch grid. Alone on the GPU, 1152-byte records move at 53-55 GB/s with 128-192
// one-wave workgroups against 49-51 GB/s with 256 (4.6 KB records: 54-55 against 53.6); inside
// the two-micro-batch decode step, beside the other micro-batch's attention, 192 workgroups
// give 1.733 ms per step against 1.748 with 256 (1152-byte records, the waves at raised issue
// priority) and the 1M-token step 2.300 against 2.324 ms, while 8 KB pages lose 0.4%.
int fetch_workgroups(const hisparse_cache_desc_t& d) {
  if (d.fetch_workgroups != 0) return d.fetch_workgroups;
  return d.record_bytes < 4096 ? 192 : 256;
}

// Staged fetch buffer layout: the per-unit prefix of entries, then the packed records.
size_t stage_rec_offset(size_t units) { return ((units + 1) * sizeof(int32_t) + 255) & ~(size_t)255; }

void free_all(hisparse_cache* c) {
  if (!c) return;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(c->device);
  (void)hipDeviceSynchronize();
  for (void* h : c->host)
    if (h) (void)hipHostFree(h);
  if (c->cache_all) (void)hipFree(c->cache_all);
  for (auto& a : c->anchors) {
    (void)hipFree(a.pt);
    (void)hipFree(a.slot_pos);
    (void)hipFree(a.slot_ts);
    (void)hipFree(a.order);
    (void)hipFree(a.clock);
    (void)hipFree(a.plan);
    (void)hipFree(a.plan_count);
    (void)hipFree(a.counts);
  }
  if (c->err) (void)hipFree(c->err);
  if (c->d_states) (void)hipFree(c->d_states);
  if (c->d_layers) (void)hipFree(c->d_layers);
  if (c->h_plan_count) (void)hipHostFree(c->h_plan_count);
  if (c->h_plan) (void)hipHostFree(c->h_plan);
  if (c->stage_done) (void)hipEventDestroy(c->stage_done);
  if (c->stage_host) (void)hipHostFree(c->stage_host);
  if (c->stage_dev) (void)hipFree(c->stage_dev);
  delete c->gather;
  (void)hipSetDevice(prev);
  delete c;
}

template <typename T>
hisparse_status_t dmalloc(T** p, size_t bytes) {
  *p = nullptr;
  if (hipMalloc(reinterpret_cast<void**>(p), bytes) != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return HISPARSE_ERR_OOM;
  }
  return HISPARSE_OK;
}

hisparse::StateArgs state_args(const hisparse_cache* c, const hisparse_cache::Anchor& a) {
  hisparse::StateArgs s{};
  s.pt = a.pt;
  s.slot_pos = a.slot_pos;
  s.slot_ts = a.slot_ts;
  s.order = a.order;
  s.clock = a.clock;
  s.plan_count = a.plan_count;
  s.L = c->desc.num_records;
  s.B = c->desc.capacity;
  s.units = c->units;
  return s;
}

// Scratch of hisparse_sparse_decode_noalloc: one array per GPU, created with the code object
// and kept until the process ends. In host code `scratch` names a host-side stand-in, not device
// memory: its device address on each GPU comes from hipGetSymbolAddress, taken once per device
// when a cache is created there.
static __device__ __align__(256) uint8_t scratch[HISPARSE_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// With `device` current: the device address of its scratch array, looked up on first use.
hisparse_status_t init_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return HISPARSE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[device]) return HISPARSE_OK;
  void* ptr = nullptr;
  if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
    (void)hipGetLastError();
    return HISPARSE_ERR_HIP;
  }
  g_scratch_ptr[device] = ptr;
  return HISPARSE_OK;
}

void* scratch_of(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return g_scratch_ptr[device];
}

}  // namespace

extern "C" {

const char* hisparse_status_string(hisparse_status_t s) {
  switch (s) {
    case HISPARSE_OK: return "HISPARSE_OK";
    case HISPARSE_ERR_INVALID_ARG: return "HISPARSE_ERR_INVALID_ARG";
    case HISPARSE_ERR_OOM: return "HISPARSE_ERR_OOM";
    case HISPARSE_ERR_HIP: return "HISPARSE_ERR_HIP";
    case HISPARSE_ERR_UNSUPPORTED: return "HISPARSE_ERR_UNSUPPORTED";
    case HISPARSE_ERR_BAD_SELECTION: return "HISPARSE_ERR_BAD_SELECTION";
    case HISPARSE_ERR_FULL: return "HISPARSE_ERR_FULL";
  }
  return "HISPARSE_ERR_UNKNOWN";
}

hisparse_status_t hisparse_validate_desc(const hisparse_cache_desc_t* d) {
  if (!d) return HISPARSE_ERR_INVALID_ARG;
  if (d->num_requests < 1 || d->num_layers < 1 || d->units_per_request < 1)
    return HISPARSE_ERR_INVALID_ARG;
  const int64_t units = (int64_t)d->num_requests * d->units_per_request;
  if (units > 65535) return HISPARSE_ERR_INVALID_ARG;
  if (d->top_k < 1 || d->top_k > kMaxTopK) return HISPARSE_ERR_INVALID_ARG;
  if (d->capacity < d->top_k || d->capacity > kMaxCapacity) return HISPARSE_ERR_INVALID_ARG;
  if (d->num_records < 1 || d->num_records > 0x7FFFFFFFLL) return HISPARSE_ERR_INVALID_ARG;
  if (d->record_bytes < 16 || d->record_bytes > kMaxRecordBytes || d->record_bytes % 16 != 0)
    return HISPARSE_ERR_INVALID_ARG;
  if (d->share_group < 1) return HISPARSE_ERR_INVALID_ARG;
  if (d->fetch != HISPARSE_FETCH_ZERO_COPY && d->fetch != HISPARSE_FETCH_SDMA &&
      d->fetch != HISPARSE_FETCH_STAGED &&
      d->fetch != HISPARSE_FETCH_NONE)
    return HISPARSE_ERR_UNSUPPORTED;
  if (d->host_memory < HISPARSE_HOST_COHERENT || d->host_memory > HISPARSE_HOST_UNCACHED)
    return HISPARSE_ERR_INVALID_ARG;
  const int tb = d->transfer_block_bytes;
  if (!(tb == 0 || tb == 16 || tb == 32 || tb == 64 || tb == 128 || tb == 256))
    return HISPARSE_ERR_INVALID_ARG;
  if (d->fetch_workgroups < 0 || d->fetch_workgroups > 4096) return HISPARSE_ERR_INVALID_ARG;
  // the resolve kernel keeps the sorted misses, the slot outputs and two slot bitmaps in LDS
  // (dynamic), beside a few hundred bytes of its own: at most a gfx950 workgroup's 160 KiB
  if (hisparse::resolve_lds_bytes(d->top_k, d->capacity) > kMaxResolveLds)
    return HISPARSE_ERR_INVALID_ARG;
  // per-unit host pool and cache offsets must fit comfortably in 64-bit byte offsets
  if ((double)d->num_records * d->record_bytes * units > 4.0e18) return HISPARSE_ERR_INVALID_ARG;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_validate_attn(int32_t record_bytes, int32_t top_k,
                                         const hisparse_attn_desc_t* a) {
  if (!a) return HISPARSE_ERR_INVALID_ARG;
  if ((a->flags & ~(HISPARSE_ATTN_DEFER_MERGE | HISPARSE_ATTN_BESIDE_FETCH |
                    HISPARSE_ATTN_CARRIES_REPLAY)) != 0 ||
      a->q_heads < 1 || a->q_heads > 256 ||
      a->num_splits < 0)
    return HISPARSE_ERR_INVALID_ARG;
  if (top_k < 1 || top_k > kMaxTopK) return HISPARSE_ERR_INVALID_ARG;
  const int tpr = a->tokens_per_record;
  if (tpr < 1 || tpr > 4096 || (tpr & (tpr - 1)) != 0) return HISPARSE_ERR_INVALID_ARG;
  if (record_bytes < 16 || record_bytes % (2 * tpr) != 0) return HISPARSE_ERR_INVALID_ARG;
  if ((int64_t)top_k * tpr > (1 << 24)) return HISPARSE_ERR_INVALID_ARG;
  const int token_elems = record_bytes / 2 / tpr;
  const bool mla = a->d_qk == 576 && a->d_v == 512 && a->v_offset == 0;
  const bool gqa = a->d_qk == 128 && a->d_v == 128 && a->v_offset == 128;
  if (!mla && !gqa) return HISPARSE_ERR_UNSUPPORTED;
  if (token_elems < std::max(a->d_qk, a->v_offset + a->d_v)) return HISPARSE_ERR_INVALID_ARG;
  // latent attention merges at most kMlaMaxParts splits of at most kMaxSplitTokens tokens
  if (mla && (int64_t)top_k * tpr > (int64_t)hisparse::kMlaMaxParts * hisparse::kMaxSplitTokens)
    return HISPARSE_ERR_UNSUPPORTED;
  if ((record_bytes / tpr) % 16 != 0) return HISPARSE_ERR_INVALID_ARG;  // 16-byte token rows
  if (!(a->scale > 0.f) || a->scale > 1e6f) return HISPARSE_ERR_INVALID_ARG;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_cache_create(const hisparse_cache_desc_t* desc, int32_t device,
                                        hisparse_cache_t* out) {
  if (!out) return HISPARSE_ERR_INVALID_ARG;
  *out = nullptr;
  hisparse_status_t st = hisparse_validate_desc(desc);
  if (st != HISPARSE_OK) return st;
  int n_dev = 0;
  if (hipGetDeviceCount(&n_dev) != hipSuccess || device < 0 || device >= n_dev) {
    (void)hipGetLastError();
    return HISPARSE_ERR_INVALID_ARG;
  }
  // the resolve kernel's LDS must also fit what this device grants one workgroup
  int max_lds = 0;
  if (hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, device) !=
      hipSuccess)
    return HISPARSE_ERR_HIP;
  if (hisparse::resolve_lds_bytes(desc->top_k, desc->capacity) + 256 > (size_t)max_lds)
    return HISPARSE_ERR_UNSUPPORTED;
  int prev = 0;
  (void)hipGetDevice(&prev);
  if (hipSetDevice(device) != hipSuccess) return HISPARSE_ERR_HIP;

  hisparse_cache* c = new (std::nothrow) hisparse_cache();
  if (!c) return HISPARSE_ERR_OOM;
  c->desc = *desc;
  c->device = device;
  c->units = desc->num_requests * desc->units_per_request;
  c->request_taken.assign(desc->num_requests, 0);
  c->n_anchors = (desc->num_layers + desc->share_group - 1) / desc->share_group;
  const size_t U = (size_t)c->units, L = (size_t)desc->num_records, B = (size_t)desc->capacity;
  const size_t R = (size_t)desc->record_bytes, K = (size_t)desc->top_k;
  c->host_layer_bytes = U * L * R;
  c->cache_layer_bytes = U * B * R;
  c->host.assign(desc->num_layers, nullptr);
  c->host_dev.assign(desc->num_layers, nullptr);
  c->cache.assign(desc->num_layers, nullptr);
  c->anchors.assign(c->n_anchors, hisparse_cache::Anchor{});

  unsigned flags = hipHostMallocMapped;
  if (desc->host_memory == HISPARSE_HOST_COHERENT) flags |= hipHostMallocCoherent;
  else if (desc->host_memory == HISPARSE_HOST_NONCOHERENT) flags |= hipHostMallocNonCoherent;
  else flags |= hipHostMallocUncached;

  st = HISPARSE_OK;
  for (int l = 0; l < desc->num_layers && st == HISPARSE_OK; ++l) {
    if (hipHostMalloc(&c->host[l], c->host_layer_bytes, flags) != hipSuccess) {
      c->host[l] = nullptr;
      (void)hipGetLastError();
      st = HISPARSE_ERR_OOM;
      break;
    }
    if (hipHostGetDevicePointer(&c->host_dev[l], c->host[l], 0) != hipSuccess) {
      (void)hipGetLastError();
      st = HISPARSE_ERR_HIP;
      break;
    }
  }
  if (st == HISPARSE_OK) {
    st = dmalloc(&c->cache_all, c->cache_layer_bytes * (size_t)desc->num_layers);
    for (int l = 0; l < desc->num_layers && st == HISPARSE_OK; ++l)
      c->cache[l] = c->cache_all + (size_t)l * c->cache_layer_bytes;
  }
  for (int a = 0; a < c->n_anchors && st == HISPARSE_OK; ++a) {
    auto& an = c->anchors[a];
    if ((st = dmalloc(&an.pt, U * L * 4)) != HISPARSE_OK) break;
    if ((st = dmalloc(&an.slot_pos, U * B * 4)) != HISPARSE_OK) break;
    if ((st = dmalloc(&an.slot_ts, U * B * 4)) != HISPARSE_OK) break;
    if ((st = dmalloc(&an.order, U * B * 4)) != HISPARSE_OK) break;
    if ((st = dmalloc(&an.clock, U * 4)) != HISPARSE_OK) break;
    if ((st = dmalloc(&an.plan, U * K * sizeof(int2))) != HISPARSE_OK) break;
    if ((st = dmalloc(&an.plan_count, U * 4)) != HISPARSE_OK) break;
    if ((st = dmalloc(&an.counts, U * 2 * 4)) != HISPARSE_OK) break;
  }
  if (st == HISPARSE_OK) st = dmalloc(&c->err, hisparse::kErrWords * 4);
  if (st == HISPARSE_OK) st = dmalloc(&c->d_states, sizeof(hisparse::AnchorState) * c->n_anchors);
  if (st == HISPARSE_OK)
    st = dmalloc(&c->d_layers, sizeof(hisparse::LayerIO) * (size_t)desc->num_layers);
  if (st == HISPARSE_OK) {
    std::vector<hisparse::AnchorState> hs_states(c->n_anchors);
    for (int a = 0; a < c->n_anchors; ++a) {
      const auto& an = c->anchors[a];
      hs_states[a] = hisparse::AnchorState{an.pt, an.slot_pos, an.slot_ts, an.order, an.clock};
    }
    std::vector<hisparse::LayerIO> hs_layers(desc->num_layers);
    for (int l = 0; l < desc->num_layers; ++l)
      hs_layers[l] = hisparse::LayerIO{c->cache[l], reinterpret_cast<uint8_t*>(c->host_dev[l])};
    if (hipMemcpy(c->d_states, hs_states.data(), sizeof(hisparse::AnchorState) * c->n_anchors,
                  hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(c->d_layers, hs_layers.data(), sizeof(hisparse::LayerIO) * desc->num_layers,
                  hipMemcpyHostToDevice) != hipSuccess)
      st = HISPARSE_ERR_HIP;
  }
  if (st == HISPARSE_OK && desc->fetch == HISPARSE_FETCH_STAGED) {
    // [units + 1] int32 prefix (256-byte aligned), then at most every unit's k records
    c->stage_bytes = stage_rec_offset(U) + U * K * R;
    if (hipHostMalloc(reinterpret_cast<void**>(&c->stage_host), c->stage_bytes, 0) !=
        hipSuccess) {
      c->stage_host = nullptr;
      (void)hipGetLastError();
      st = HISPARSE_ERR_OOM;
    } else {
      st = dmalloc(&c->stage_dev, c->stage_bytes);
    }
    if (st == HISPARSE_OK &&
        hipEventCreateWithFlags(&c->stage_done, hipEventDisableTiming) != hipSuccess) {
      c->stage_done = nullptr;
      st = HISPARSE_ERR_HIP;
    }
    if (st == HISPARSE_OK) {
      c->gather = new (std::nothrow) hisparse::GatherPool(hisparse::GatherPool::host_threads(16));
      if (!c->gather) st = HISPARSE_ERR_OOM;
    }
  }
  if (st == HISPARSE_OK &&
      (desc->fetch == HISPARSE_FETCH_SDMA || desc->fetch == HISPARSE_FETCH_STAGED)) {
    if (hipHostMalloc(reinterpret_cast<void**>(&c->h_plan_count), U * 4, 0) != hipSuccess ||
        hipHostMalloc(reinterpret_cast<void**>(&c->h_plan), U * K * sizeof(int2), 0) !=
            hipSuccess) {
      (void)hipGetLastError();
      st = HISPARSE_ERR_OOM;
    } else {
      c->dma_dst.resize(U * K);
      c->dma_src.resize(U * K);
      c->dma_size.resize(U * K);
    }
  }
  if (st == HISPARSE_OK) {
    if (hipMemset(c->err, 0, hisparse::kErrWords * 4) != hipSuccess) st = HISPARSE_ERR_HIP;
    if (hipMemset(c->cache_all, 0, c->cache_layer_bytes * (size_t)desc->num_layers) != hipSuccess)
      st = HISPARSE_ERR_HIP;
    for (int a = 0; a < c->n_anchors && st == HISPARSE_OK; ++a) {
      if (hipMemset(c->anchors[a].plan, 0xFF, U * K * sizeof(int2)) != hipSuccess ||
          hisparse::launch_reset_state(state_args(c, c->anchors[a]), nullptr) != hipSuccess)
        st = HISPARSE_ERR_HIP;
    }
    if (st == HISPARSE_OK && hipDeviceSynchronize() != hipSuccess) st = HISPARSE_ERR_HIP;
  }
  // the allocation-free attention's scratch on this device (once per device)
  if (st == HISPARSE_OK) st = init_scratch(device);
  (void)hipSetDevice(prev);
  if (st != HISPARSE_OK) {
    (void)hipGetLastError();
    free_all(c);
    return st;
  }
  *out = c;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_cache_destroy(hisparse_cache_t c) {
  free_all(c);
  return HISPARSE_OK;
}

hisparse_status_t hisparse_host_pool(hisparse_cache_t c, int32_t layer, void** host,
                                     size_t* bytes) {
  if (!c || layer < 0 || layer >= c->desc.num_layers) return HISPARSE_ERR_INVALID_ARG;
  if (host) *host = c->host[layer];
  if (bytes) *bytes = c->host_layer_bytes;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_layer_cache(hisparse_cache_t c, int32_t layer, void** device,
                                       size_t* bytes) {
  if (!c || layer < 0 || layer >= c->desc.num_layers) return HISPARSE_ERR_INVALID_ARG;
  if (device) *device = c->cache[layer];
  if (bytes) *bytes = c->cache_layer_bytes;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_reset(hisparse_cache_t c, void* stream) {
  if (!c) return HISPARSE_ERR_INVALID_ARG;
  for (auto& a : c->anchors)
    if (hisparse::launch_reset_state(state_args(c, a), as_stream(stream)) != hipSuccess)
      return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_reset_units(hisparse_cache_t c, int32_t first_unit, int32_t num_units,
                                       void* stream) {
  if (!c || first_unit < 0 || num_units < 1 || num_units > c->units - first_unit)
    return HISPARSE_ERR_INVALID_ARG;
  const int64_t L = c->desc.num_records, B = c->desc.capacity;
  for (auto& a : c->anchors) {
    hisparse::StateArgs s = state_args(c, a);  // the same cold-state kernel on a unit range
    s.pt += first_unit * L;
    s.slot_pos += first_unit * B;
    s.slot_ts += first_unit * B;
    s.order += first_unit * B;
    s.clock += first_unit;
    s.plan_count += first_unit;
    s.units = num_units;
    if (hisparse::launch_reset_state(s, as_stream(stream)) != hipSuccess) return HISPARSE_ERR_HIP;
  }
  return HISPARSE_OK;
}

hisparse_status_t hisparse_request_acquire(hisparse_cache_t c, int32_t* request) {
  if (!c || !request) return HISPARSE_ERR_INVALID_ARG;
  *request = -1;
  for (size_t r = 0; r < c->request_taken.size(); ++r)
    if (!c->request_taken[r]) {
      c->request_taken[r] = 1;
      *request = (int32_t)r;
      return HISPARSE_OK;
    }
  return HISPARSE_ERR_FULL;
}

hisparse_status_t hisparse_request_release(hisparse_cache_t c, int32_t request, void* stream) {
  if (!c || request < 0 || request >= c->desc.num_requests || !c->request_taken[request])
    return HISPARSE_ERR_INVALID_ARG;
  const int32_t H = c->desc.units_per_request;
  const hisparse_status_t st = hisparse_reset_units(c, request * H, H, stream);
  if (st == HISPARSE_OK) c->request_taken[request] = 0;
  return st;
}

hisparse_status_t hisparse_stage(hisparse_cache_t c, int32_t first_layer, int32_t num_layers,
                                 int32_t first_unit, int32_t num_units, int64_t first_record,
                                 int64_t num_records, const void* d_src,
                                 int64_t src_layer_stride, void* stream) {
  if (!c || !d_src || first_layer < 0 || num_layers < 1 ||
      num_layers > c->desc.num_layers - first_layer || first_unit < 0 || num_units < 1 ||
      num_units > c->units - first_unit)
    return HISPARSE_ERR_INVALID_ARG;
  const int64_t L = c->desc.num_records, R = c->desc.record_bytes;
  if (first_record < 0 || num_records < 1 || num_records > L - first_record)
    return HISPARSE_ERR_INVALID_ARG;
  const int64_t unit_bytes = num_records * R, layer_bytes = num_units * unit_bytes;
  if (num_layers > 1 && src_layer_stride < layer_bytes) return HISPARSE_ERR_INVALID_ARG;
  const bool whole = num_records == L || num_units == 1;  // one contiguous range per layer
  for (int32_t j = 0; j < num_layers; ++j) {
    const uint8_t* src = reinterpret_cast<const uint8_t*>(d_src) + j * src_layer_stride;
    uint8_t* dst = reinterpret_cast<uint8_t*>(c->host[first_layer + j]) +
                   ((int64_t)first_unit * L + first_record) * R;
    for (int32_t u = 0; u < (whole ? 1 : num_units); ++u)
      if (hipMemcpyAsync(dst + u * L * R, src + u * unit_bytes,
                         (size_t)(whole ? layer_bytes : unit_bytes), hipMemcpyDeviceToHost,
                         as_stream(stream)) != hipSuccess)
        return HISPARSE_ERR_HIP;
  }
  return HISPARSE_OK;
}

hisparse_status_t hisparse_append(hisparse_cache_t c, int32_t first_layer, int32_t num_layers,
                                  const int32_t* d_pos, const void* d_records, int32_t* d_slots,
                                  void* stream) {
  if (!c || !d_pos || !d_records || !d_slots || !is_anchor(c, first_layer) || num_layers < 1 ||
      num_layers > c->desc.num_layers - first_layer)
    return HISPARSE_ERR_INVALID_ARG;
  const int32_t G = c->desc.share_group, end = first_layer + num_layers;
  if (end % G != 0 && end != c->desc.num_layers) return HISPARSE_ERR_INVALID_ARG;  // whole groups
  hisparse::AdmitArgs a{};
  a.pos = d_pos;
  a.states = c->d_states;
  a.layers = c->d_layers;
  a.records = reinterpret_cast<const uint8_t*>(d_records);
  a.slots_out = d_slots;
  a.err = c->err;
  a.L = c->desc.num_records;
  a.B = c->desc.capacity;
  a.R = c->desc.record_bytes;
  a.units = c->units;
  a.G = G;
  a.first = first_layer;
  a.n_layers = num_layers;
  a.write = c->desc.fetch != HISPARSE_FETCH_NONE;  // NONE: tables only, no record moved
  if (hisparse::launch_admit(a, (num_layers + G - 1) / G, as_stream(stream)) != hipSuccess)
    return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}

namespace {
// Phases 1-3 and 5 of an anchor layer; d_slots may be null (no slot vector is written).
hisparse_status_t resolve_tables(hisparse_cache_t c, int32_t layer, const int32_t* d_sel,
                                 int32_t* d_slots, int32_t* d_counts, void* stream) {
  auto& an = c->anchors[layer / c->desc.share_group];
  hisparse::ResolveArgs a{};
  a.sel = d_sel;
  a.pt = an.pt;
  a.slot_pos = an.slot_pos;
  a.slot_ts = an.slot_ts;
  a.order = an.order;
  a.clock = an.clock;
  a.slots_out = d_slots;
  a.counts_out = d_counts ? d_counts : an.counts;
  a.plan = an.plan;
  a.plan_count = an.plan_count;
  a.err = c->err;
  a.L = c->desc.num_records;
  a.B = c->desc.capacity;
  a.k = c->desc.top_k;
  a.layer = layer;
  a.units = c->units;
  if (hisparse::launch_resolve(a, as_stream(stream)) != hipSuccess) return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}
}  // namespace

hisparse_status_t hisparse_resolve_tables(hisparse_cache_t c, int32_t layer,
                                          const int32_t* d_sel, int32_t* d_slots,
                                          int32_t* d_counts, void* stream) {
  if (!c || !d_sel || !d_slots || !is_anchor(c, layer)) return HISPARSE_ERR_INVALID_ARG;
  return resolve_tables(c, layer, d_sel, d_slots, d_counts, stream);
}

namespace {
// Kernel arguments for copying `anchor`'s latest miss plan into target layers [target, target +
// n_layers) (n_layers <= kMaxFetchLayers), units [u0, u0 + nu).
hisparse::FetchArgs fetch_args(hisparse_cache_t c, int32_t anchor, int32_t target, int32_t u0,
                               int32_t nu, int32_t n_layers) {
  auto& an = c->anchors[anchor / c->desc.share_group];
  const int64_t L = c->desc.num_records, B = c->desc.capacity, R = c->desc.record_bytes;
  hisparse::FetchArgs f{};
  f.n_layers = n_layers;
  f.plan = an.plan + (int64_t)u0 * c->desc.top_k;
  f.plan_count = an.plan_count + u0;
  for (int32_t j = 0; j < n_layers; ++j)
    f.host[j] = reinterpret_cast<const uint8_t*>(c->host_dev[target + j]) + (int64_t)u0 * L * R;
  f.cache = c->cache[target] + (int64_t)u0 * B * R;
  f.cache_stride = (int64_t)c->cache_layer_bytes;
  f.L = L;
  f.B = (int32_t)B;
  f.k = c->desc.top_k;
  f.R = (int32_t)R;
  f.units = nu;
  f.part_lo = 0;
  f.part_hi = 256;
  return f;
}

// Copy the records of `anchor`'s latest miss plan from each target layer's host pool into
// its GPU cache, for targets [target, target + n_layers) and units [u0, u0 + nu) (target ==
// anchor: the demand fetch; a shared layer: the prefetch replay).
// Entries [m * part_lo / 256, m * part_hi / 256) of each unit's plan of m entries only.
hisparse_status_t enqueue_fetch(hisparse_cache_t c, int32_t anchor, int32_t target,
                                hipStream_t stream, int32_t u0 = 0, int32_t nu = -1,
                                int32_t n_layers = 1, int32_t part_lo = 0,
                                int32_t part_hi = 256,
                                const hisparse::LinkTurn* turn = nullptr) {
  if (nu < 0) nu = c->units - u0;
  if (c->desc.fetch == HISPARSE_FETCH_NONE || nu == 0 || part_lo >= part_hi) return HISPARSE_OK;
  if ((c->desc.fetch == HISPARSE_FETCH_SDMA || c->desc.fetch == HISPARSE_FETCH_STAGED) &&
      n_layers > 1) {
    for (int32_t j = 0; j < n_layers; ++j) {
      const hisparse_status_t st =
          enqueue_fetch(c, anchor, target + j, stream, u0, nu, 1, part_lo, part_hi);
      if (st != HISPARSE_OK) return st;
    }
    return HISPARSE_OK;
  }
  auto& an = c->anchors[anchor / c->desc.share_group];
  if (c->desc.fetch == HISPARSE_FETCH_STAGED) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess) return HISPARSE_ERR_HIP;
    if (cs != hipStreamCaptureStatusNone) return HISPARSE_ERR_UNSUPPORTED;
    const size_t U = (size_t)c->units, K = (size_t)c->desc.top_k;
    // The staging buffers are the handle's: the previous staged fetch, on whatever stream,
    // must have copied out of the pinned one and scattered out of the device one before this
    // one refills them (an event never recorded is complete).
    if (hipEventSynchronize(c->stage_done) != hipSuccess) return HISPARSE_ERR_HIP;
    // the plan, once the resolve that wrote it has run
    if (hipMemcpyAsync(c->h_plan_count, an.plan_count, U * 4, hipMemcpyDeviceToHost, stream) !=
            hipSuccess ||
        hipMemcpyAsync(c->h_plan, an.plan, U * K * sizeof(int2), hipMemcpyDeviceToHost,
                       stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
      return HISPARSE_ERR_HIP;
    const size_t R = (size_t)c->desc.record_bytes, L = (size_t)c->desc.num_records;
    int32_t* prefix = reinterpret_cast<int32_t*>(c->stage_host);
    // entries of the range per unit; prefix[u] = first packed entry of unit u
    std::vector<int32_t> lo(U, 0);
    int32_t n = 0;
    for (size_t u = 0; u < U; ++u) {
      const int32_t m = c->h_plan_count[u];
      const bool in = u >= (size_t)u0 && u < (size_t)u0 + (size_t)nu;
      lo[u] = (m * part_lo) >> 8;
      prefix[u] = n;
      if (in) n += ((m * part_hi) >> 8) - lo[u];
    }
    prefix[U] = n;
    if (n == 0) return HISPARSE_OK;
    const size_t off = stage_rec_offset(U);
    uint8_t* rec = c->stage_host + off;
    const uint8_t* host = reinterpret_cast<const uint8_t*>(c->host[target]);
    const int2* plan = c->h_plan;
    if (hipMemcpyAsync(c->stage_dev, c->stage_host, off, hipMemcpyHostToDevice, stream) !=
        hipSuccess)
      return HISPARSE_ERR_HIP;
    // The worker threads gather the records in increasing order, in pieces of about 1 MiB;
    // this thread enqueues each piece's copy as soon as the piece is packed, so the copy
    // engine moves one piece while the workers gather the next (with no worker thread, this
    // thread gathers everything first).
    constexpr int64_t kGrain = 16;  // entries per hand-out; a piece is a whole number of them
    const int64_t piece = std::max<int64_t>(4, (int64_t)((1 << 20) / R) / kGrain) * kGrain;
    const int64_t n_pieces = (n + piece - 1) / piece;
    std::vector<std::atomic<int64_t>> packed(n_pieces);
    for (auto& x : packed) x.store(0);
    const std::function<void(int64_t, int64_t)> gather = [&](int64_t b, int64_t e) {
      size_t u = std::upper_bound(prefix, prefix + U + 1, (int32_t)b) - prefix - 1;
      for (int64_t j = b; j < e; ++j) {
        while (j >= prefix[u + 1]) ++u;
        const int2 pe = plan[u * K + lo[u] + (j - prefix[u])];
        memcpy(rec + (size_t)j * R, host + (u * L + (size_t)pe.x) * R, R);
      }
      packed[b / piece].fetch_add(e - b, std::memory_order_release);
    };
    const bool async = c->gather->threads() > 1;
    if (async) c->gather->start(n, kGrain, gather);
    else c->gather->run(n, kGrain, gather);
    hisparse_status_t copy_st = HISPARSE_OK;
    for (int64_t q = 0; q < n_pieces; ++q) {
      const int64_t p0 = q * piece, p1 = std::min<int64_t>(n, p0 + piece);
      while (packed[q].load(std::memory_order_acquire) < p1 - p0) std::this_thread::yield();
      if (copy_st == HISPARSE_OK &&
          hipMemcpyAsync(c->stage_dev + off + (size_t)p0 * R, rec + (size_t)p0 * R,
                         (size_t)(p1 - p0) * R, hipMemcpyHostToDevice, stream) != hipSuccess)
        copy_st = HISPARSE_ERR_HIP;
    }
    if (async) c->gather->wait();
    if (copy_st != HISPARSE_OK) return copy_st;
    // the scatter reads each unit's range of the plan: the same entries, in plan order
    hisparse::ScatterArgs sa{};
    sa.stage = c->stage_dev;
    sa.plan = an.plan;
    sa.cache = c->cache[target];
    sa.rec_offset = (int64_t)stage_rec_offset(U);
    sa.B = c->desc.capacity;
    sa.k = c->desc.top_k;
    sa.R = c->desc.record_bytes;
    sa.units = c->units;
    sa.plan_count = an.plan_count;
    sa.part_lo = part_lo;
    if (hisparse::launch_scatter(sa, stream) != hipSuccess ||
        hipEventRecord(c->stage_done, stream) != hipSuccess)
      return HISPARSE_ERR_HIP;
    return HISPARSE_OK;
  }
  if (c->desc.fetch == HISPARSE_FETCH_SDMA) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess) return HISPARSE_ERR_HIP;
    if (cs != hipStreamCaptureStatusNone) return HISPARSE_ERR_UNSUPPORTED;
    const size_t U = (size_t)c->units, K = (size_t)c->desc.top_k;
    if (hipMemcpyAsync(c->h_plan_count, an.plan_count, U * 4, hipMemcpyDeviceToHost, stream) !=
            hipSuccess ||
        hipMemcpyAsync(c->h_plan, an.plan, U * K * sizeof(int2), hipMemcpyDeviceToHost,
                       stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
      return HISPARSE_ERR_HIP;
    const size_t u_end = (size_t)u0 + (size_t)nu;
    const size_t R = (size_t)c->desc.record_bytes, L = (size_t)c->desc.num_records;
    const size_t B = (size_t)c->desc.capacity;
    uint8_t* host = reinterpret_cast<uint8_t*>(c->host[target]);
    uint8_t* cache = c->cache[target];
    size_t n = 0;
    for (size_t u = (size_t)u0; u < u_end; ++u) {
      const int2* pl = c->h_plan + u * K;
      const int32_t m = c->h_plan_count[u];
      for (int32_t i = (m * part_lo) >> 8; i < (m * part_hi) >> 8; ++i) {
        uint8_t* src = host + (u * L + (size_t)pl[i].x) * R;
        uint8_t* dst = cache + (u * B + (size_t)pl[i].y) * R;
        if (n && (uint8_t*)c->dma_src[n - 1] + c->dma_size[n - 1] == src &&
            (uint8_t*)c->dma_dst[n - 1] + c->dma_size[n - 1] == dst) {
          c->dma_size[n - 1] += R;  // adjacent positions into adjacent slots: one copy
        } else {
          c->dma_src[n] = src;
          c->dma_dst[n] = dst;
          c->dma_size[n] = R;
          ++n;
        }
      }
    }
    if (n == 0) return HISPARSE_OK;
    if (batch_copy_fn fn = batch_copy()) {
      // one copy-engine batch; a runtime that refuses the call (e.g. wants explicit copy
      // attributes) gets the copies one by one below instead
      hipMemcpyAttributes attr;
      memset(&attr, 0, sizeof(attr));
      attr.srcAccessOrder = hipMemcpySrcAccessOrderStream;  // sources read in stream order
      attr.srcLocHint.type = hipMemLocationTypeHost;
      attr.dstLocHint.type = hipMemLocationTypeDevice;
      attr.dstLocHint.id = c->device;
      size_t attr_idx = 0, fail = 0;
      if (fn(c->dma_dst.data(), c->dma_src.data(), c->dma_size.data(), n, &attr, &attr_idx, 1,
             &fail, stream) == hipSuccess)
        return HISPARSE_OK;
      (void)hipGetLastError();
    }
    for (size_t i = 0; i < n; ++i)
      if (hipMemcpyAsync(c->dma_dst[i], c->dma_src[i], c->dma_size[i], hipMemcpyHostToDevice,
                         stream) != hipSuccess)
        return HISPARSE_ERR_HIP;
    return HISPARSE_OK;
  }
  for (int32_t j0 = 0; j0 < n_layers; j0 += hisparse::kMaxFetchLayers) {
    hisparse::FetchArgs f = fetch_args(c, anchor, target + j0, u0, nu,
                                       std::min(n_layers - j0, hisparse::kMaxFetchLayers));
    f.part_lo = part_lo;
    f.part_hi = part_hi;
    if (hisparse::launch_fetch(f, transfer_block(c->desc), fetch_workgroups(c->desc), stream,
                               turn) != hipSuccess)
      return HISPARSE_ERR_HIP;
  }
  return HISPARSE_OK;
}
}  // namespace

hisparse_status_t hisparse_fetch(hisparse_cache_t c, int32_t layer, void* stream) {
  if (!c || !is_anchor(c, layer)) return HISPARSE_ERR_INVALID_ARG;
  return enqueue_fetch(c, layer, layer, as_stream(stream));
}

hisparse_status_t hisparse_fetch_part(hisparse_cache_t c, int32_t layer, int32_t part_begin,
                                      int32_t part_end, void* stream) {
  if (!c || !is_anchor(c, layer) || part_begin < 0 || part_begin > part_end || part_end > 256)
    return HISPARSE_ERR_INVALID_ARG;
  return enqueue_fetch(c, layer, layer, as_stream(stream), 0, -1, 1, part_begin, part_end);
}

hisparse_status_t hisparse_fetch_turn(hisparse_cache_t c, int32_t layer, int32_t* d_turns,
                                      int32_t n_turns, int32_t wait_turn, int32_t signal_turn,
                                      int32_t signal_share, void* stream) {
  if (!c || !is_anchor(c, layer) || !d_turns || n_turns < 1 || wait_turn < -1 ||
      signal_turn < -1 || wait_turn >= n_turns || signal_turn >= n_turns || signal_share < 1 ||
      signal_share > 256 || (wait_turn >= 0 && wait_turn == signal_turn))
    return HISPARSE_ERR_INVALID_ARG;
  // host-issued copies and no-IO caches have no kernel to take a turn (a waiting launch would
  // run out its bound)
  if (c->desc.fetch != HISPARSE_FETCH_ZERO_COPY) return HISPARSE_ERR_UNSUPPORTED;
  const hisparse::LinkTurn t{d_turns, wait_turn, signal_turn, signal_share};
  return enqueue_fetch(c, layer, layer, as_stream(stream), 0, -1, 1, 0, 256, &t);
}

hisparse_status_t hisparse_link_turns_reset(int32_t* d_turns, int32_t n_turns, void* stream) {
  if (!d_turns || n_turns < 1 || n_turns > (1 << 24)) return HISPARSE_ERR_INVALID_ARG;
  return hisparse::launch_turns_reset(d_turns, n_turns, as_stream(stream)) == hipSuccess
             ? HISPARSE_OK
             : HISPARSE_ERR_HIP;
}

hisparse_status_t hisparse_fetch_units(hisparse_cache_t c, int32_t layer, int32_t unit_begin,
                                       int32_t unit_count, void* stream) {
  if (!c || !is_anchor(c, layer) || unit_begin < 0 || unit_count < 0 ||
      unit_count > c->units - unit_begin)
    return HISPARSE_ERR_INVALID_ARG;
  return enqueue_fetch(c, layer, layer, as_stream(stream), unit_begin, unit_count);
}

hisparse_status_t hisparse_fetch_group(hisparse_cache_t c, int32_t anchor_layer,
                                       int32_t num_layers, void* stream) {
  if (!c || !is_anchor(c, anchor_layer) || num_layers < 1 ||
      num_layers > c->desc.share_group || num_layers > c->desc.num_layers - anchor_layer)
    return HISPARSE_ERR_INVALID_ARG;
  return enqueue_fetch(c, anchor_layer, anchor_layer, as_stream(stream), 0, -1, num_layers);
}

hisparse_status_t hisparse_resolve(hisparse_cache_t c, int32_t layer, const int32_t* d_sel,
                                   int32_t* d_slots, int32_t* d_counts, void* stream) {
  hisparse_status_t st = hisparse_resolve_tables(c, layer, d_sel, d_slots, d_counts, stream);
  if (st != HISPARSE_OK) return st;
  return enqueue_fetch(c, layer, layer, as_stream(stream));
}

hisparse_status_t hisparse_speculate(hisparse_cache_t c, int32_t layer, const int32_t* d_hint,
                                     int32_t* d_counts, void* stream) {
  if (!c || !d_hint || !is_anchor(c, layer)) return HISPARSE_ERR_INVALID_ARG;
  hisparse_status_t st = resolve_tables(c, layer, d_hint, nullptr, d_counts, stream);
  if (st != HISPARSE_OK) return st;
  return enqueue_fetch(c, layer, layer, as_stream(stream));
}

hisparse_status_t hisparse_prefetch_layer(hisparse_cache_t c, int32_t anchor_layer,
                                          int32_t shared_layer, void* stream) {
  if (!c || !is_anchor(c, anchor_layer)) return HISPARSE_ERR_INVALID_ARG;
  if (shared_layer <= anchor_layer || shared_layer >= c->desc.num_layers ||
      shared_layer - anchor_layer >= c->desc.share_group)
    return HISPARSE_ERR_INVALID_ARG;
  return enqueue_fetch(c, anchor_layer, shared_layer, as_stream(stream));
}

hisparse_status_t hisparse_prefetch_layers(hisparse_cache_t c, int32_t anchor_layer,
                                           int32_t first_shared, int32_t num_layers,
                                           void* stream) {
  if (!c || !is_anchor(c, anchor_layer) || num_layers < 1) return HISPARSE_ERR_INVALID_ARG;
  const int64_t end = (int64_t)first_shared + num_layers;
  if (first_shared <= anchor_layer ||
      end > std::min<int64_t>((int64_t)anchor_layer + c->desc.share_group, c->desc.num_layers))
    return HISPARSE_ERR_INVALID_ARG;
  return enqueue_fetch(c, anchor_layer, first_shared, as_stream(stream), 0, -1, num_layers);
}

size_t hisparse_decode_workspace_bytes(int32_t units, int32_t top_k, int32_t record_bytes,
                                       const hisparse_attn_desc_t* attn) {
  hisparse::AttnPlan p{};
  if (hisparse::plan_attention(units, top_k, record_bytes, attn, &p) != HISPARSE_OK) return 0;
  return p.workspace_bytes;
}

hisparse_status_t hisparse_sparse_decode_pool(const void* d_pool, int64_t records_per_unit,
                                              int32_t record_bytes, int32_t units, int32_t top_k,
                                              const void* d_q, const int32_t* d_idx, float* d_out,
                                              const hisparse_attn_desc_t* attn,
                                              void* d_workspace, size_t workspace_bytes,
                                              void* stream) {
  if (!d_pool || !d_q || !d_idx || !d_out || !d_workspace || records_per_unit < 1)
    return HISPARSE_ERR_INVALID_ARG;
  hisparse::AttnPlan p{};
  hisparse_status_t st = hisparse::plan_attention(units, top_k, record_bytes, attn, &p);
  if (st != HISPARSE_OK) return st;
  if (workspace_bytes < p.workspace_bytes) return HISPARSE_ERR_INVALID_ARG;
  // the kernel addresses a unit's records with 32-bit byte offsets
  if (records_per_unit * (int64_t)record_bytes > (int64_t)INT32_MAX) return HISPARSE_ERR_UNSUPPORTED;
  if (hisparse::launch_attention(p, *attn, reinterpret_cast<const uint8_t*>(d_pool),
                                 records_per_unit, record_bytes, units, top_k,
                                 reinterpret_cast<const uint16_t*>(d_q), d_idx, d_out, d_workspace,
                                 as_stream(stream)) != hipSuccess)
    return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_attention_merge(int32_t units, int32_t top_k, int32_t record_bytes,
                                           const hisparse_attn_desc_t* attn, float* d_out,
                                           const void* d_workspace, size_t workspace_bytes,
                                           void* stream) {
  if (!d_out || !d_workspace) return HISPARSE_ERR_INVALID_ARG;
  hisparse::AttnPlan p{};
  hisparse_status_t st = hisparse::plan_attention(units, top_k, record_bytes, attn, &p);
  if (st != HISPARSE_OK) return st;
  if (workspace_bytes < p.workspace_bytes) return HISPARSE_ERR_INVALID_ARG;
  if (hisparse::launch_merge(p, *attn, units, d_out, d_workspace, as_stream(stream)) !=
      hipSuccess)
    return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_sparse_decode(hisparse_cache_t c, int32_t layer, const void* d_q,
                                         const int32_t* d_slots, float* d_out,
                                         const hisparse_attn_desc_t* attn, void* d_workspace,
                                         size_t workspace_bytes, void* stream) {
  if (!c || layer < 0 || layer >= c->desc.num_layers) return HISPARSE_ERR_INVALID_ARG;
  return hisparse_sparse_decode_pool(c->cache[layer], c->desc.capacity, c->desc.record_bytes,
                                     c->units, c->desc.top_k, d_q, d_slots, d_out, attn,
                                     d_workspace, workspace_bytes, stream);
}

hisparse_status_t hisparse_sparse_decode_noalloc(hisparse_cache_t c, int32_t layer,
                                                 const void* d_q, const int32_t* d_slots,
                                                 float* d_out, const hisparse_attn_desc_t* attn,
                                                 void* stream) {
  if (!c || layer < 0 || layer >= c->desc.num_layers) return HISPARSE_ERR_INVALID_ARG;
  if (!d_q || !d_slots || !d_out || !attn) return HISPARSE_ERR_INVALID_ARG;
  // the split partials must be merged within the call: nothing else can find them
  if (attn->flags & HISPARSE_ATTN_DEFER_MERGE) return HISPARSE_ERR_INVALID_ARG;
  hisparse::AttnPlan p{};
  hisparse_status_t st =
      hisparse::plan_attention(c->units, c->desc.top_k, c->desc.record_bytes, attn, &p);
  if (st != HISPARSE_OK) return st;
  if (p.workspace_bytes > HISPARSE_NOALLOC_SCRATCH_BYTES) return HISPARSE_ERR_UNSUPPORTED;
  if ((int64_t)c->desc.capacity * c->desc.record_bytes > (int64_t)INT32_MAX)
    return HISPARSE_ERR_UNSUPPORTED;
  void* ws = scratch_of(c->device);
  if (!ws) return HISPARSE_ERR_HIP;
  if (hisparse::launch_attention(p, *attn, c->cache[layer], c->desc.capacity,
                                 c->desc.record_bytes, c->units, c->desc.top_k,
                                 reinterpret_cast<const uint16_t*>(d_q), d_slots, d_out, ws,
                                 as_stream(stream)) != hipSuccess)
    return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}

namespace {
// Checks of a replay of `anchor_layer`'s plan into shared layers [first_shared, first_shared +
// num_shared) over plan-entry range [part_begin, part_end) in 256ths.
bool valid_replay(hisparse_cache_t c, int32_t anchor_layer, int32_t first_shared,
                  int32_t num_shared, int32_t part_begin, int32_t part_end) {
  if (!is_anchor(c, anchor_layer) || num_shared < 1 || num_shared > hisparse::kMaxFetchLayers)
    return false;
  const int64_t end = (int64_t)first_shared + num_shared;
  if (first_shared <= anchor_layer ||
      end > std::min<int64_t>((int64_t)anchor_layer + c->desc.share_group, c->desc.num_layers))
    return false;
  return 0 <= part_begin && part_begin <= part_end && part_end <= 256;
}
}  // namespace

hisparse_status_t hisparse_sparse_decode_prefetch_part(
    hisparse_cache_t c, int32_t layer, const void* d_q, const int32_t* d_slots, float* d_out,
    const hisparse_attn_desc_t* attn, void* d_workspace, size_t workspace_bytes,
    int32_t anchor_layer, int32_t first_shared, int32_t num_shared, int32_t part_begin,
    int32_t part_end, void* stream) {
  if (!c || layer < 0 || layer >= c->desc.num_layers) return HISPARSE_ERR_INVALID_ARG;
  if (!valid_replay(c, anchor_layer, first_shared, num_shared, part_begin, part_end))
    return HISPARSE_ERR_INVALID_ARG;
  if (layer >= first_shared && layer < first_shared + num_shared)
    return HISPARSE_ERR_INVALID_ARG;  // reads what it writes
  if (!d_q || !d_slots || !d_out || !d_workspace) return HISPARSE_ERR_INVALID_ARG;
  if (c->desc.fetch != HISPARSE_FETCH_ZERO_COPY) {
    // no kernel-issued copy to carry: the replay on its own (or nothing), then the attention
    const hisparse_status_t st = enqueue_fetch(c, anchor_layer, first_shared, as_stream(stream),
                                               0, -1, num_shared, part_begin, part_end);
    if (st != HISPARSE_OK) return st;
    return hisparse_sparse_decode(c, layer, d_q, d_slots, d_out, attn, d_workspace,
                                  workspace_bytes, stream);
  }
  hisparse::AttnPlan p{};
  hisparse_status_t st =
      hisparse::plan_attention(c->units, c->desc.top_k, c->desc.record_bytes, attn, &p);
  if (st != HISPARSE_OK) return st;
  if (workspace_bytes < p.workspace_bytes) return HISPARSE_ERR_INVALID_ARG;
  if ((int64_t)c->desc.capacity * c->desc.record_bytes > (int64_t)INT32_MAX)
    return HISPARSE_ERR_UNSUPPORTED;
  hisparse::FetchArgs f = fetch_args(c, anchor_layer, first_shared, 0, c->units, num_shared);
  f.part_lo = part_begin;
  f.part_hi = part_end;
  if (hisparse::launch_attention(p, *attn, c->cache[layer], c->desc.capacity,
                                 c->desc.record_bytes, c->units, c->desc.top_k,
                                 reinterpret_cast<const uint16_t*>(d_q), d_slots, d_out,
                                 d_workspace, as_stream(stream), 0,
                                 part_begin < part_end ? &f : nullptr,
                                 fetch_workgroups(c->desc) * 64 * 2,
                                 transfer_block(c->desc) * 2) != hipSuccess)
    return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_sparse_decode_prefetch(hisparse_cache_t c, int32_t layer,
                                                  const void* d_q, const int32_t* d_slots,
                                                  float* d_out, const hisparse_attn_desc_t* attn,
                                                  void* d_workspace, size_t workspace_bytes,
                                                  int32_t anchor_layer, int32_t first_shared,
                                                  int32_t num_shared, void* stream) {
  return hisparse_sparse_decode_prefetch_part(c, layer, d_q, d_slots, d_out, attn, d_workspace,
                                              workspace_bytes, anchor_layer, first_shared,
                                              num_shared, 0, 256, stream);
}

hisparse_status_t hisparse_attention_merge_prefetch(hisparse_cache_t c,
                                                    const hisparse_attn_desc_t* attn,
                                                    float* d_out, const void* d_workspace,
                                                    size_t workspace_bytes, int32_t anchor_layer,
                                                    int32_t first_shared, int32_t num_shared,
                                                    int32_t part_begin, int32_t part_end,
                                                    void* stream) {
  if (!c || !d_out || !d_workspace) return HISPARSE_ERR_INVALID_ARG;
  if (!valid_replay(c, anchor_layer, first_shared, num_shared, part_begin, part_end))
    return HISPARSE_ERR_INVALID_ARG;
  hisparse::AttnPlan p{};
  hisparse_status_t st =
      hisparse::plan_attention(c->units, c->desc.top_k, c->desc.record_bytes, attn, &p);
  if (st != HISPARSE_OK) return st;
  if (workspace_bytes < p.workspace_bytes) return HISPARSE_ERR_INVALID_ARG;
  if (c->desc.fetch != HISPARSE_FETCH_ZERO_COPY) {
    st = enqueue_fetch(c, anchor_layer, first_shared, as_stream(stream), 0, -1, num_shared,
                       part_begin, part_end);
    if (st != HISPARSE_OK) return st;
    return hisparse::launch_merge(p, *attn, c->units, d_out, d_workspace, as_stream(stream)) ==
                   hipSuccess
               ? HISPARSE_OK
               : HISPARSE_ERR_HIP;
  }
  hisparse::FetchArgs f = fetch_args(c, anchor_layer, first_shared, 0, c->units, num_shared);
  f.part_lo = part_begin;
  f.part_hi = part_end;
  if (hisparse::launch_merge(p, *attn, c->units, d_out, d_workspace, as_stream(stream),
                             part_begin < part_end ? &f : nullptr,
                             fetch_workgroups(c->desc) * 64 * 2,
                             transfer_block(c->desc) * 2) != hipSuccess)
    return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_sparse_decode_layers(hisparse_cache_t c, int32_t first_layer,
                                                int32_t num_layers, const void* d_q,
                                                const int32_t* d_slots, float* d_out,
                                                const hisparse_attn_desc_t* attn,
                                                void* d_workspace, size_t workspace_bytes,
                                                void* stream) {
  if (!c || first_layer < 0 || num_layers < 1 || num_layers > c->desc.num_layers - first_layer)
    return HISPARSE_ERR_INVALID_ARG;
  const int G = c->desc.share_group;
  if (first_layer / G != (first_layer + num_layers - 1) / G) return HISPARSE_ERR_INVALID_ARG;
  if (!d_q || !d_slots || !d_out || !d_workspace) return HISPARSE_ERR_INVALID_ARG;
  if ((int64_t)c->units * num_layers > (int64_t)INT32_MAX / 256) return HISPARSE_ERR_INVALID_ARG;
  const int32_t units = c->units * num_layers;
  hisparse::AttnPlan p{};
  hisparse_status_t st =
      hisparse::plan_attention(units, c->desc.top_k, c->desc.record_bytes, attn, &p);
  if (st != HISPARSE_OK) return st;
  if (workspace_bytes < p.workspace_bytes) return HISPARSE_ERR_INVALID_ARG;
  if ((int64_t)c->desc.capacity * c->desc.record_bytes > (int64_t)INT32_MAX)
    return HISPARSE_ERR_UNSUPPORTED;
  // the layers' caches are consecutive in one allocation, so unit u of layer first + j is
  // unit j * units + u of one pool; every layer reads the same slot vector
  if (hisparse::launch_attention(p, *attn, c->cache[first_layer], c->desc.capacity,
                                 c->desc.record_bytes, units, c->desc.top_k,
                                 reinterpret_cast<const uint16_t*>(d_q), d_slots, d_out,
                                 d_workspace, as_stream(stream), c->units) != hipSuccess)
    return HISPARSE_ERR_HIP;
  return HISPARSE_OK;
}

hisparse_status_t hisparse_read_state(hisparse_cache_t c, int32_t layer, int32_t* slot_pos,
                                      uint32_t* slot_ts, int32_t* page_table, int32_t* order,
                                      uint32_t* clock) {
  if (!c || !is_anchor(c, layer)) return HISPARSE_ERR_INVALID_ARG;
  auto& an = c->anchors[layer / c->desc.share_group];
  const size_t U = (size_t)c->units, B = (size_t)c->desc.capacity;
  const size_t L = (size_t)c->desc.num_records;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(c->device);
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess && slot_pos) e = hipMemcpy(slot_pos, an.slot_pos, U * B * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess && slot_ts) e = hipMemcpy(slot_ts, an.slot_ts, U * B * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess && page_table) e = hipMemcpy(page_table, an.pt, U * L * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess && order) e = hipMemcpy(order, an.order, U * B * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess && clock) e = hipMemcpy(clock, an.clock, U * 4, hipMemcpyDeviceToHost);
  (void)hipSetDevice(prev);
  return e == hipSuccess ? HISPARSE_OK : HISPARSE_ERR_HIP;
}

hisparse_status_t hisparse_read_plan(hisparse_cache_t c, int32_t layer, int32_t* plan,
                                     int32_t* count) {
  if (!c || !is_anchor(c, layer)) return HISPARSE_ERR_INVALID_ARG;
  auto& an = c->anchors[layer / c->desc.share_group];
  const size_t U = (size_t)c->units, K = (size_t)c->desc.top_k;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(c->device);
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess && plan) e = hipMemcpy(plan, an.plan, U * K * sizeof(int2), hipMemcpyDeviceToHost);
  if (e == hipSuccess && count) e = hipMemcpy(count, an.plan_count, U * 4, hipMemcpyDeviceToHost);
  (void)hipSetDevice(prev);
  return e == hipSuccess ? HISPARSE_OK : HISPARSE_ERR_HIP;
}

hisparse_status_t hisparse_check_errors(hisparse_cache_t c, int32_t* info) {
  if (!c) return HISPARSE_ERR_INVALID_ARG;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(c->device);
  int32_t w[hisparse::kErrWords] = {0, 0, 0, 0};
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(w, c->err, sizeof(w), hipMemcpyDeviceToHost);
  if (e == hipSuccess && w[0] != 0) e = hipMemset(c->err, 0, sizeof(w));
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return HISPARSE_ERR_HIP;
  if (info) {
    info[0] = w[1];
    info[1] = w[2];
    info[2] = w[3];
  }
  return w[0] != 0 ? (hisparse_status_t)w[0] : HISPARSE_OK;
}

hisparse_status_t hisparse_debug_resolve_phases(uint64_t* host_stamps, int32_t max_units,
                                                int64_t* ticks_per_s) {
#ifndef HISPARSE_PHASE_STAMPS
  (void)host_stamps;
  (void)max_units;
  (void)ticks_per_s;
  return HISPARSE_ERR_UNSUPPORTED;
#else
  if (!host_stamps || max_units <= 0) return HISPARSE_ERR_INVALID_ARG;
  const int32_t n = std::min<int32_t>(max_units, hisparse::kPhaseStampUnits);
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceSynchronize() != hipSuccess ||
      hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      hisparse::read_resolve_phase_stamps(host_stamps, n) != hipSuccess)
    return HISPARSE_ERR_HIP;
  if (ticks_per_s) *ticks_per_s = (int64_t)khz * 1000;
  return HISPARSE_OK;
#endif
}

}  // extern "C"
