// HiSparse resolve (Section 3.4 phases 1-3 and 5) and miss fetch (phase 4) for gfx950.
//
// resolve_kernel: one workgroup per cache unit.
//   Phase 1  stage the unit's selection: validate entries, probe the page table for each
//            (k gathers instead of the paper's probe of all B slots against a hash: the
//            position->slot table answers membership directly), mark hit slots in an LDS
//            bitmap (a second mark on the same slot is a repeated entry), and append the
//            misses as (position, input index) keys to LDS.
//   Phase 2  sort the miss keys (LDS bitonic sort): ascending position order is what the
//            canonical victim pairing needs, and equal neighbours expose repeated misses.
//   Phase 3  victims and recency: the unit keeps a recency index `order` = its slots sorted
//            by (timestamp, slot). Victims are the first m entries of `order` that were not
//            hit (one workgroup prefix scan); the new index is
//              [kept entries in old order] ++ [victims by slot] ++ [hits by slot],
//            which is exactly the sort by the new (timestamp, slot) because every new stamp
//            (2t-1 for misses, 2t for hits) exceeds every old one.
//   Phase 5  update page table / slot map / stamps, record the miss plan, and publish the
//            slot of every input entry in input order.
// fetch_kernel: copies each planned record from the pinned host pool (zero-copy 16-byte
//   loads through the mapped address) into its slot; a wide grid over all units' misses, so a
//   layer call with few units still keeps many loads in flight across the chip.
#include "internal.h"

namespace hisparse {
namespace {

constexpr int kWave = 64;
constexpr int kMaxChunk = 16;  // order entries per thread: B <= 16 * threads

__device__ inline int wave_incl_scan(int x, int lane) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  return x;
}

// Exclusive workgroup scan of v; *total = sum over the workgroup. s_tmp: NT/64 + 1 ints.
// Starts and ends with a barrier-protected use of s_tmp.
template <int NT>
__device__ inline int block_excl_scan(int v, int* s_tmp, int* total) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const int incl = wave_incl_scan(v, lane);
  if (lane == kWave - 1) s_tmp[wid] = incl;
  __syncthreads();
  if (wid == 0) {
    const int w = lane < NW ? s_tmp[lane] : 0;
    const int wi = wave_incl_scan(w, lane);
    if (lane < NW) s_tmp[lane] = wi - w;
    if (lane == NW - 1) s_tmp[NW] = wi;
  }
  __syncthreads();
  const int r = s_tmp[wid] + incl - v;
  *total = s_tmp[NW];
  __syncthreads();
  return r;
}

// Ascending bitonic sort of n (a power of two) 64-bit keys in LDS.
template <int NT>
__device__ inline void bitonic_sort(uint64_t* keys, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int idx = threadIdx.x; idx < (n >> 1); idx += NT) {
        const int lo = ((idx & ~(stride - 1)) << 1) | (idx & (stride - 1));
        const int hi = lo + stride;
        const bool asc = (lo & size) == 0;
        const uint64_t x = keys[lo], y = keys[hi];
        if ((x > y) == asc) {
          keys[lo] = y;
          keys[hi] = x;
        }
      }
      __syncthreads();
    }
  }
}

__host__ __device__ inline int pow2_at_least(int n) {
  int p = 2;
  while (p < n) p <<= 1;
  return p;
}

__device__ inline bool bit_test(const uint32_t* bm, int s) { return (bm[s >> 5] >> (s & 31)) & 1u; }

template <int NT>
__global__ __launch_bounds__(NT) void resolve_kernel(ResolveArgs a) {
  extern __shared__ __align__(16) unsigned char s_dyn[];
  __shared__ int s_tmp[NT / kWave + 1];
  __shared__ int s_nmiss, s_bad;

  const int unit = blockIdx.x;
  const int tid = threadIdx.x;
  const int k = a.k, B = a.B;
  const int64_t L = a.L;
  const int p2k = pow2_at_least(k);
  const int k4 = (k + 3) & ~3;
  const int bw = (B + 31) >> 5;

  uint64_t* s_keys = reinterpret_cast<uint64_t*>(s_dyn);   // [p2k] miss keys (pos << 32 | i)
  int32_t* s_out = reinterpret_cast<int32_t*>(s_keys + p2k);  // [k4] slot per input index
  int32_t* s_victim = s_out + k4;                           // [k4] victim slot per miss rank
  uint32_t* s_hit = reinterpret_cast<uint32_t*>(s_victim + k4);  // [bw] slots hit this step
  uint32_t* s_vic = s_hit + bw;                             // [bw] slots taken as victims

  const int32_t* sel = a.sel + (int64_t)unit * k;
  int32_t* pt = a.pt + (int64_t)unit * L;
  int32_t* slot_pos = a.slot_pos + (int64_t)unit * B;
  uint32_t* slot_ts = a.slot_ts + (int64_t)unit * B;
  int32_t* order = a.order + (int64_t)unit * B;
  int32_t* slots_out = a.slots_out + (int64_t)unit * k;
  int2* plan = a.plan + (int64_t)unit * k;

  for (int i = tid; i < bw; i += NT) {
    s_hit[i] = 0u;
    s_vic[i] = 0u;
  }
  if (tid == 0) {
    s_nmiss = 0;
    s_bad = 0;
  }
  __syncthreads();

  // Phase 1: stage, validate, probe.
  for (int i = tid; i < k; i += NT) {
    const int32_t p = sel[i];
    int32_t out = -1;
    if (p >= 0) {
      if ((int64_t)p >= L) {
        s_bad = 1;
      } else {
        const int32_t s = pt[p];
        if (s >= 0) {
          const uint32_t bit = 1u << (s & 31);
          if (atomicOr(&s_hit[s >> 5], bit) & bit) s_bad = 1;  // repeated resident entry
          out = s;
        } else {
          const int r = atomicAdd(&s_nmiss, 1);
          s_keys[r] = ((uint64_t)(uint32_t)p << 32) | (uint32_t)i;
        }
      }
    }
    s_out[i] = out;
  }
  __syncthreads();
  const int m = s_nmiss;

  // Phase 2: misses in ascending position order; repeated misses become neighbours.
  const int p2 = pow2_at_least(m);
  for (int i = m + tid; i < p2; i += NT) s_keys[i] = ~0ull;
  __syncthreads();
  bitonic_sort<NT>(s_keys, p2);
  for (int r = 1 + tid; r < m; r += NT)
    if ((s_keys[r] >> 32) == (s_keys[r - 1] >> 32)) s_bad = 1;
  __syncthreads();

  if (s_bad) {  // invalid selection: publish -1 and leave the unit's state untouched
    for (int i = tid; i < k; i += NT) slots_out[i] = -1;
    if (tid == 0) {
      if (a.counts_out) {
        a.counts_out[2 * unit] = 0;
        a.counts_out[2 * unit + 1] = 0;
      }
      a.plan_count[unit] = 0;
      if (atomicCAS(&a.err[0], 0, (int)HISPARSE_ERR_BAD_SELECTION) == 0) {
        a.err[1] = a.layer;
        a.err[2] = unit;
      }
      atomicAdd(&a.err[3], 1);
    }
    return;
  }

  const uint32_t t = a.clock[unit] + 1u;

  // Phase 3a: victims = first m non-hit entries of the recency index.
  const int ch = (B + NT - 1) / NT;
  const int j0 = tid * ch;
  int32_t ov[kMaxChunk];
  int cnt = 0;
#pragma unroll
  for (int c = 0; c < kMaxChunk; ++c) {
    ov[c] = -1;
    if (c < ch && j0 + c < B) {
      ov[c] = order[j0 + c];
      cnt += bit_test(s_hit, ov[c]) ? 0 : 1;
    }
  }
  int total_nonhit;
  int r = block_excl_scan<NT>(cnt, s_tmp, &total_nonhit);  // all reads of `order` precede it
#pragma unroll
  for (int c = 0; c < kMaxChunk; ++c) {
    const int32_t s = ov[c];
    if (s >= 0 && !bit_test(s_hit, s)) {
      if (r < m) {
        s_victim[r] = s;
        atomicOr(&s_vic[s >> 5], 1u << (s & 31));
      } else {
        order[r - m] = s;  // kept entries slide to the least-recent end
      }
      ++r;
    }
  }
  __syncthreads();

  // Phase 3b: recency index tail (victims, then hits, each by slot) and hit stamps.
  int nv = 0, nh = 0;
#pragma unroll
  for (int c = 0; c < kMaxChunk; ++c) {
    const int s = j0 + c;
    if (c < ch && s < B) {
      nv += bit_test(s_vic, s) ? 1 : 0;
      nh += bit_test(s_hit, s) ? 1 : 0;
    }
  }
  int packed_total;
  const int base = block_excl_scan<NT>((nv << 16) | nh, s_tmp, &packed_total);
  const int hits = packed_total & 0xFFFF;
  int rv = base >> 16, rh = base & 0xFFFF;
  const uint32_t ts_hit = 2u * t, ts_miss = 2u * t - 1u;
#pragma unroll
  for (int c = 0; c < kMaxChunk; ++c) {
    const int s = j0 + c;
    if (c < ch && s < B) {
      if (bit_test(s_vic, s)) {
        order[B - hits - m + rv++] = s;
      } else if (bit_test(s_hit, s)) {
        order[B - hits + rh++] = s;
        slot_ts[s] = ts_hit;
      }
    }
  }

  // Phase 5: the i-th miss (ascending position) takes the i-th victim.
  for (int q = tid; q < m; q += NT) {
    const uint64_t key = s_keys[q];
    const int32_t p = (int32_t)(key >> 32);
    const int32_t i = (int32_t)(key & 0xFFFFFFFFu);
    const int32_t v = s_victim[q];
    const int32_t old = slot_pos[v];
    if (old >= 0) pt[old] = -1;  // evicted record becomes host-only
    pt[p] = v;
    slot_pos[v] = p;
    slot_ts[v] = ts_miss;
    plan[q] = make_int2(p, v);
    s_out[i] = v;
  }
  __syncthreads();
  for (int i = tid; i < k; i += NT) slots_out[i] = s_out[i];
  if (tid == 0) {
    if (a.counts_out) {
      a.counts_out[2 * unit] = hits;
      a.counts_out[2 * unit + 1] = m;
    }
    a.plan_count[unit] = m;
    a.clock[unit] = t;
  }
}

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

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int U>
__global__ __launch_bounds__(256) void fetch_kernel(FetchArgs a, FastDiv div_cpr) {
  const int unit = blockIdx.y;
  const int m = a.plan_count[unit];
  const uint32_t cpr = (uint32_t)a.R >> 4;  // 16-byte chunks per record
  const uint32_t total = (uint32_t)m * cpr;
  const int2* plan = a.plan + (int64_t)unit * a.k;
  const uint8_t* host = a.host + (int64_t)unit * a.L * a.R;
  uint8_t* cache = a.cache + (int64_t)unit * a.B * a.R;
  const uint32_t stride = gridDim.x * 256u;
  for (uint32_t c0 = blockIdx.x * 256u + threadIdx.x; c0 < total; c0 += stride * U) {
    u32x4 v[U];
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
            reinterpret_cast<const u32x4*>(host + (int64_t)pe.x * a.R + (w << 4)));
        dst[u] = (int64_t)pe.y * a.R + (w << 4);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (dst[u] >= 0) *reinterpret_cast<u32x4*>(cache + dst[u]) = v[u];
  }
}

__global__ void reset_state_kernel(StateArgs a) {
  const int64_t n_pt = (int64_t)a.units * a.L;
  const int64_t n_slots = (int64_t)a.units * a.B;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_pt; i += stride)
    a.pt[i] = -1;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_slots; i += stride) {
    a.slot_pos[i] = -1;
    a.slot_ts[i] = 0u;
    a.order[i] = (int32_t)(i % a.B);
  }
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.units; i += stride) {
    a.clock[i] = 0u;
    a.plan_count[i] = 0;
  }
}

template <int NT>
hipError_t launch_resolve_nt(const ResolveArgs& a, size_t lds, hipStream_t stream) {
  hipLaunchKernelGGL(resolve_kernel<NT>, dim3(a.units), dim3(NT), lds, stream, a);
  return hipGetLastError();
}

}  // namespace

size_t resolve_lds_bytes(int32_t k, int32_t B) {
  const size_t k4 = (size_t)((k + 3) & ~3);
  return 8 * (size_t)pow2_at_least(k) + 8 * k4 + 8 * (size_t)((B + 31) >> 5);
}

hipError_t launch_resolve(const ResolveArgs& a, hipStream_t stream) {
  const size_t lds = resolve_lds_bytes(a.k, a.B);
  int nt = 64;
  while (nt < 1024 && nt * kMaxChunk < a.B) nt <<= 1;
  while (nt < 1024 && nt * 4 < a.B) nt <<= 1;  // about four order entries per thread
  switch (nt) {
    case 64: return launch_resolve_nt<64>(a, lds, stream);
    case 128: return launch_resolve_nt<128>(a, lds, stream);
    case 256: return launch_resolve_nt<256>(a, lds, stream);
    case 512: return launch_resolve_nt<512>(a, lds, stream);
    default: return launch_resolve_nt<1024>(a, lds, stream);
  }
}

hipError_t launch_fetch(const FetchArgs& a, int transfer_block_bytes, hipStream_t stream) {
  const int U = transfer_block_bytes / 16;
  const int64_t max_chunks = (int64_t)a.k * (a.R / 16);
  int64_t x = (max_chunks + 256LL * U - 1) / (256LL * U);
  const int64_t cap = std::max<int64_t>(1, 4096 / a.units);
  if (x > cap) x = cap;
  const dim3 grid((unsigned)x, (unsigned)a.units);
  const FastDiv f = make_fastdiv((uint32_t)(a.R / 16));
  switch (U) {
    case 1: hipLaunchKernelGGL(fetch_kernel<1>, grid, dim3(256), 0, stream, a, f); break;
    case 2: hipLaunchKernelGGL(fetch_kernel<2>, grid, dim3(256), 0, stream, a, f); break;
    case 4: hipLaunchKernelGGL(fetch_kernel<4>, grid, dim3(256), 0, stream, a, f); break;
    case 8: hipLaunchKernelGGL(fetch_kernel<8>, grid, dim3(256), 0, stream, a, f); break;
    default: hipLaunchKernelGGL(fetch_kernel<16>, grid, dim3(256), 0, stream, a, f); break;
  }
  return hipGetLastError();
}

hipError_t launch_reset_state(const StateArgs& a, hipStream_t stream) {
  const int64_t n = std::max<int64_t>((int64_t)a.units * a.L, (int64_t)a.units * a.B);
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(reset_state_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace hisparse
