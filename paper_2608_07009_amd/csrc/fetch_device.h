// Device side of the miss fetch (Section 3.4 Phase 4) and of the exact-prefetch replay
// (Section 3.5), shared by the standalone fetch kernel and by the attention kernels that carry
// a replay in the same launch.
#pragma once

#include "internal.h"

namespace hisparse {

// Unsigned division by a runtime constant d >= 1 for n < 2^31 (round-up multiplier method:
// magic = floor(2^32 (2^l - d) / d) + 1, l = ceil(log2 d); n / d = (umulhi(n, magic) + n) >> l).
struct FastDiv {
  uint32_t magic, shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  uint64_t magic = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
  return FastDiv{(uint32_t)magic, l};
}

__device__ inline uint32_t fastdiv(uint32_t n, FastDiv f) {
  return (__umulhi(n, f.magic) + n) >> f.shift;
}

// One thread's share of copying unit `unit`'s planned records into target layer z: the 16-byte
// chunks first, first + stride, ... of the plan's entry range (chunk c = 16-byte piece
// c % (R / 16) of plan entry c / (R / 16)), U loads in flight before their stores. Each planned
// record is read from the layer's host pool at its position and written to the layer's cache at
// its slot.
template <int U>
__device__ __forceinline__ void fetch_slice(const FetchArgs& a, FastDiv div_cpr, int unit, int z,
                                            uint32_t first, uint32_t stride) {
  typedef unsigned int v4u __attribute__((ext_vector_type(4)));
  const int m = a.plan_count[unit];
  const uint32_t cpr = (uint32_t)a.R >> 4;  // 16-byte chunks per record
  const uint32_t total = (uint32_t)((m * a.part_hi) >> 8) * cpr;
  first += (uint32_t)((m * a.part_lo) >> 8) * cpr;
  const int2* plan = a.plan + (int64_t)unit * a.k;
  const uint8_t* host = a.host[z] + (int64_t)unit * a.L * a.R;
  uint8_t* cache = a.cache + (int64_t)z * a.cache_stride + (int64_t)unit * a.B * a.R;
  for (uint32_t c0 = first; c0 < total; c0 += stride * U) {
    v4u v[U];
    int64_t dst[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t c = c0 + u * stride;
      dst[u] = -1;
      if (c < total) {
        const uint32_t r = fastdiv(c, div_cpr);
        const uint32_t w = c - r * cpr;
        const int2 pe = plan[r];
        v[u] = __builtin_nontemporal_load(
            reinterpret_cast<const v4u*>(host + (int64_t)pe.x * a.R + (w << 4)));
        dst[u] = (int64_t)pe.y * a.R + (w << 4);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (dst[u] >= 0) *reinterpret_cast<v4u*>(cache + dst[u]) = v[u];
  }
}

}  // namespace hisparse
