// HiSparse resolve (Section 3.4 phases 1-3 and 5) and miss fetch (phase 4) for gfx950.
//
// resolve_kernel: one workgroup per cache unit.
//   Phase 1  stage the unit's selection: validate entries, probe the page table for each
//            (k gathers instead of the paper's probe of all B slots against a hash: the
//            position->slot table answers membership directly), mark hit slots in an LDS
//            bitmap (a second mark on the same slot is a repeated entry), and append the
//            misses as (position, input index) keys to LDS.
//   Phase 2  put the miss keys in ascending position order (what the canonical victim
//            pairing needs): a counting pass over up to 2048 buckets of high position bits
//            (twice the misses, at least 64, when there are at most 256) gives each bucket's
//            start, and a miss's rank is its bucket start plus the number of bucket mates at
//            lower positions; a mate at the same position exposes a repeated miss. A few
//            barriers in all, where a sorting network needs dozens.
//   Phase 3  victims and recency: the unit keeps a recency index `order` = its slots sorted
//            by (timestamp, slot). Victims are the first m entries of `order` that were not
//            hit (one workgroup prefix scan); the new index is
//              [kept entries in old order] ++ [victims by slot] ++ [hits by slot],
//            which is exactly the sort by the new (timestamp, slot) because every new stamp
//            (2t-1 for misses, 2t for hits) exceeds every old one.
//   Phase 5  update page table / slot map / stamps, record the miss plan, and publish the
//            slot of every input entry in input order.
// fetch_kernel: copies each planned record from the pinned host pool (zero-copy 16-byte
//   loads through the mapped address) into its slot. The grid is small: a fixed budget of
//   one-wave workgroups shared by the launch's units, each thread keeping one transfer block
//   of loads in flight. A few hundred KB of reads in flight saturate the host link; spread
//   thinly over the chip, the fetch keeps only a few slow host reads outstanding per CU,
//   which limits how much it delays other streams' work on the same CUs. One launch can
//   serve several layers of a share group (grid z): the anchor's demand fetch and the
//   replays of the same plan into its shared layers.
#include "fetch_device.h"

namespace hisparse {
namespace {

constexpr int kWave = 64;
constexpr int kMaxChunk = 16;  // order entries per thread: B <= 16 * threads
constexpr int kMaxPer = 4;     // selections per thread: k <= 4 * threads
constexpr int kBucketBits = 11;
constexpr int kBuckets = 1 << kBucketBits;  // miss rank buckets (high position bits)
// The most misses one rank bucket may hold before the misses are sorted instead of counted
// (counting mates costs about bucket size x misses per thread steps per thread).
#ifndef HISPARSE_SCAN_LIMIT
constexpr int kScanLimit = 256;
#else
constexpr int kScanLimit = HISPARSE_SCAN_LIMIT;
#endif
// One wave per fetch workgroup: each CU that hosts fetch work gives it one wave and a few
// outstanding host reads, not a whole workgroup's worth.
constexpr int kFetchThreads = 64;

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


__device__ inline bool bit_test(const uint32_t* bm, int s) { return (bm[s >> 5] >> (s & 31)) & 1u; }

#ifdef HISPARSE_PHASE_STAMPS
__device__ unsigned long long g_phase_stamps[kPhaseStampUnits * kPhaseStamps];
// Phase-timing build: thread 0 of the workgroups of the first kPhaseStampUnits units stores the
// constant-rate wall clock at each phase boundary (plain vector stores); the host reads the
// last launch's stamps with hisparse_debug_resolve_phases. Normal builds compile none of it.
#define RESOLVE_STAMP(i)                                                                   \
  do {                                                                                     \
    if (tid == 0 && unit < kPhaseStampUnits)                                               \
      g_phase_stamps[unit * kPhaseStamps + (i)] = (unsigned long long)wall_clock64();      \
  } while (0)
#define RESOLVE_STAMP_BARRIER() __syncthreads()
#else
#define RESOLVE_STAMP(i) \
  do {                   \
  } while (0)
#define RESOLVE_STAMP_BARRIER() \
  do {                          \
  } while (0)
#endif

template <int NT>
__global__ __launch_bounds__(NT) void resolve_kernel(ResolveArgs a) {
  extern __shared__ __align__(16) unsigned char s_dyn[];
  __shared__ int s_tmp[NT / kWave + 1];
  __shared__ int s_nmiss, s_bad;
  __shared__ int s_pmin, s_pmax, s_maxb;  // miss position range, largest bucket

  const int unit = blockIdx.x;
  const int tid = threadIdx.x;
  RESOLVE_STAMP(0);
  const int k = a.k, B = a.B;
  const int64_t L = a.L;
  const int k4 = (k + 3) & ~3;
  const int bw = (B + 31) >> 5;

  uint64_t* s_keys = reinterpret_cast<uint64_t*>(s_dyn);   // [k4] miss keys (pos << 32 | i)
  int32_t* s_out = reinterpret_cast<int32_t*>(s_keys + k4);  // [k4] slot per input index
  int32_t* s_victim = s_out + k4;                           // [k4] victim slot per miss rank
  uint32_t* s_hit = reinterpret_cast<uint32_t*>(s_victim + k4);  // [bw] slots hit this step
  uint32_t* s_vic = s_hit + bw;                             // [bw] slots taken as victims
  int32_t* s_cnt = reinterpret_cast<int32_t*>(s_vic + bw);  // [kBuckets] miss rank buckets

  const int32_t* sel = a.sel + (int64_t)unit * k;
  int32_t* pt = a.pt + (int64_t)unit * L;
  int32_t* slot_pos = a.slot_pos + (int64_t)unit * B;
  uint32_t* slot_ts = a.slot_ts + (int64_t)unit * B;
  int32_t* order = a.order + (int64_t)unit * B;
  int32_t* slots_out = a.slots_out ? a.slots_out + (int64_t)unit * k : nullptr;  // null: no slot vector
  int2* plan = a.plan + (int64_t)unit * k;

  for (int i = tid; i < bw; i += NT) {
    s_hit[i] = 0u;
    s_vic[i] = 0u;
  }
  if (tid == 0) {
    s_nmiss = 0;
    s_bad = 0;
    s_pmin = INT32_MAX;
    s_pmax = -1;
    s_maxb = 0;
  }
  __syncthreads();

  // Phase 1: stage, validate, probe. A thread handles at most kMaxPer selections (k <= 4 NT);
  // all its selection reads, then all its page-table probes, are issued before any is used.
  int32_t pv[kMaxPer], sv[kMaxPer];
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int i = tid + u * NT;
    pv[u] = i < k ? sel[i] : -1;
  }
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) sv[u] = (pv[u] >= 0 && (int64_t)pv[u] < L) ? pt[pv[u]] : -1;
  int pmin = INT32_MAX, pmax = -1;  // this thread's miss positions (phase 2 buckets by them)
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int i = tid + u * NT;
    if (i < k) {
      const int32_t p = pv[u], s = sv[u];
      int32_t out = -1;
      if (p >= 0) {
        if ((int64_t)p >= L) {
          s_bad = 1;
        } else if (s >= 0) {
          const uint32_t bit = 1u << (s & 31);
          if (atomicOr(&s_hit[s >> 5], bit) & bit) s_bad = 1;  // repeated resident entry
          out = s;
        } else {
          const int r = atomicAdd(&s_nmiss, 1);
          s_keys[r] = ((uint64_t)(uint32_t)p << 32) | (uint32_t)i;
          pmin = min(pmin, p);
          pmax = max(pmax, p);
        }
      }
      s_out[i] = out;
    }
  }
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    pmin = min(pmin, __shfl_xor(pmin, o, kWave));
    pmax = max(pmax, __shfl_xor(pmax, o, kWave));
  }
  if ((tid & (kWave - 1)) == 0 && pmax >= 0) {  // one LDS atomic pair per wave
    atomicMin(&s_pmin, pmin);
    atomicMax(&s_pmax, pmax);
  }
  // rank buckets cleared here for large workgroups (a few stores per thread beside the probes'
  // latency), after the miss count for small ones (which then need a barrier of their own)
  if constexpr (NT >= 256)
    for (int b = tid; b < kBuckets; b += NT) s_cnt[b] = 0;
  __syncthreads();
  const int m = s_nmiss;
  RESOLVE_STAMP(1);
  // rank buckets: twice the misses (at least 64) for up to 256 misses, so that a few misses
  // do not pay for a scan over all kBuckets; kBuckets beyond
  const int nbb = m <= 32 ? 6 : (m <= 256 ? 33 - __clz(m - 1) : kBucketBits);
  const int nb = 1 << nbb;
  if constexpr (NT < 256) {
    for (int b = tid; b < nb; b += NT) s_cnt[b] = 0;
    __syncthreads();
  }

  // Phase 2: the misses in ascending position order. Bucket them by the high bits of their
  // offset within the misses' own position range (a counting pass), then each miss's rank is
  // its bucket's start plus the number of bucket mates at lower positions; a mate at the same
  // position is a repeated selection. Positions are distinct, so a bucket holds at most its
  // width in misses: a contiguous run of misses spreads over the buckets. Should some bucket
  // still hold more than kScanLimit misses (clusters far apart), counting mates would cost more
  // than sorting, and the keys are sorted instead (bitonic network in LDS).
  uint64_t key[kMaxPer];
  int bkt[kMaxPer], loc[kMaxPer];
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int j = tid + u * NT;
    key[u] = j < m ? s_keys[j] : 0ull;
  }
  pmin = s_pmin;
  const uint32_t span = s_pmax > pmin ? (uint32_t)(s_pmax - pmin) : 0u;  // < 2^31
  const int lg = span ? 32 - __clz(span) : 0;
  const int shift = lg > nbb ? lg - nbb : 0;
  const uint32_t low_mask = (1u << shift) - 1u;
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int j = tid + u * NT;
    bkt[u] = j < m ? (int)((uint32_t)((int)(key[u] >> 32) - pmin) >> shift) : 0;
    loc[u] = j < m ? atomicAdd(&s_cnt[bkt[u]], 1) : 0;
  }
  __syncthreads();
  RESOLVE_STAMP(2);
  {
    // exclusive scan of the bucket counts, nb / NT consecutive buckets per thread (one for
    // threads below nb when nb <= NT)
    constexpr int kPer = (kBuckets + NT - 1) / NT;
    const int per = nb > NT ? nb / NT : 1;
    int c[kPer], sum = 0, big = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int b = tid * per + q;
      c[q] = (q < per && b < nb) ? s_cnt[b] : 0;
      sum += c[q];
      big = max(big, c[q]);
    }
    if (big > kScanLimit) atomicMax(&s_maxb, big);
    int total;
    int run = block_excl_scan<NT>(sum, s_tmp, &total);  // all reads of s_cnt precede it
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int b = tid * per + q;
      if (q < per && b < nb) s_cnt[b] = run;
      run += c[q];
    }
  }
  __syncthreads();
  RESOLVE_STAMP(3);
  if (s_maxb > kScanLimit) {  // workgroup-uniform
    // bitonic sort of the m keys in place, ascending (position, input index); the network's
    // comparators all put the smaller key at the lower index, so indices >= m act as +inf
    // padding and are never touched
    int n2 = 1;
    while (n2 < m) n2 <<= 1;
    for (int size = 2; size <= n2; size <<= 1) {
      for (int stride = size >> 1; stride >= 1; stride >>= 1) {
        for (int c = tid; c < (n2 >> 1); c += NT) {
          int i, j;
          if (stride == (size >> 1)) {  // first step of a merge: mirrored pairs
            const int blk = c / stride, off = c - blk * stride;
            i = blk * size + off;
            j = blk * size + size - 1 - off;
          } else {
            i = (c / stride) * 2 * stride + c % stride;
            j = i + stride;
          }
          if (j < m) {
            const uint64_t x = s_keys[i], y = s_keys[j];
            if (y < x) {
              s_keys[i] = y;
              s_keys[j] = x;
            }
          }
        }
        __syncthreads();
      }
    }
    for (int q = tid; q + 1 < m; q += NT)
      if ((s_keys[q] >> 32) == (s_keys[q + 1] >> 32)) s_bad = 1;  // a repeated miss
    __syncthreads();
  } else {
    // bucketed order in the victim array (free until phase 3): low offset bits and input index
    uint32_t* s_bkt = reinterpret_cast<uint32_t*>(s_victim);
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u)
      if (tid + u * NT < m)
        s_bkt[s_cnt[bkt[u]] + loc[u]] =
            ((((uint32_t)((int)(key[u] >> 32) - pmin)) & low_mask) << 12) | (uint32_t)key[u];
    __syncthreads();
    int rank[kMaxPer];
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u) {
      rank[u] = 0;
      if (tid + u * NT < m) {
        const int b0 = s_cnt[bkt[u]];
        const int b1 = bkt[u] + 1 < nb ? s_cnt[bkt[u] + 1] : m;
        const uint32_t mine = ((uint32_t)((int)(key[u] >> 32) - pmin)) & low_mask;
        const uint32_t me = (uint32_t)key[u] & 0xFFFu;
        int lower = 0;
        bool rep = false;
        int q = b0;
        for (; q + 4 <= b1; q += 4) {  // four mates' reads in flight
          uint32_t e[4];
#pragma unroll
          for (int x = 0; x < 4; ++x) e[x] = s_bkt[q + x];
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            lower += (e[x] >> 12) < mine ? 1 : 0;
            rep |= (e[x] >> 12) == mine && (e[x] & 0xFFFu) != me;
          }
        }
        for (; q < b1; ++q) {
          const uint32_t e = s_bkt[q];
          lower += (e >> 12) < mine ? 1 : 0;
          rep |= (e >> 12) == mine && (e & 0xFFFu) != me;
        }
        if (rep) s_bad = 1;
        rank[u] = b0 + lower;
      }
    }
    __syncthreads();  // all reads of the unsorted keys are done
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u)
      if (tid + u * NT < m) s_keys[rank[u]] = key[u];
    __syncthreads();
  }

  RESOLVE_STAMP(4);
  if (s_bad) {  // invalid selection: publish -1 and leave the unit's state untouched
    if (slots_out)
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
  RESOLVE_STAMP(5);

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
  RESOLVE_STAMP_BARRIER();
  RESOLVE_STAMP(6);

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
  RESOLVE_STAMP(7);
  if (slots_out)
    for (int i = tid; i < k; i += NT) slots_out[i] = s_out[i];
  if (tid == 0) {
    if (a.counts_out) {
      a.counts_out[2 * unit] = hits;
      a.counts_out[2 * unit + 1] = m;
    }
    a.plan_count[unit] = m;
    a.clock[unit] = t;
  }
  RESOLVE_STAMP(8);
}

// Link turns as the fetch kernel sees them: the turn to wait for before reading and the turn
// to signal (null: none), and the count of finished workgroups that opens the next turn. A
// turn's word 0 counts the signalling launch's finished workgroups; word 1 is 0 until that
// launch has started, 1 once it has, 2 once the waiting launch may read.
struct TurnDev {
  const int32_t* wait_pair;
  int32_t* signal_pair;
  int32_t go;
};

// A turn only orders the launches' use of the host link; no launch reads what another writes,
// so a wait that outlasts its bound simply proceeds: a signalling launch that has started is
// waited for up to kTurnWaitTicks, one that has not (not yet dispatched, or queued behind the
// waiter) up to kTurnStartTicks. Issued in turn order, a signalling launch starts before its
// waiter or within microseconds of it.
constexpr uint64_t kTurnWaitTicks = 400000;  // 4 ms of the constant 100 MHz clock
constexpr uint64_t kTurnStartTicks = 5000;   // 50 us

template <int U>
__global__ __launch_bounds__(kFetchThreads) void fetch_kernel(FetchArgs a, FastDiv div_cpr,
                                                              TurnDev turn) {
  // The fetch shares its CUs with other streams' kernels (the other micro-batch's attention and
  // merge); its waves issue little but each issue keeps the host link fed, so they go first.
  __builtin_amdgcn_s_setprio(3);
  if (turn.signal_pair && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 &&
      threadIdx.x == 0)
    __hip_atomic_fetch_max(turn.signal_pair + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (turn.wait_pair) {
    // Waves of a launch that waits for its turn are resident already and poll its state (an
    // uncached device-scope read every few hundred cycles), so the link passes from one launch
    // to the next without a dependency through the command processor.
    const uint64_t t0 = wall_clock64();
    for (;;) {
      const int32_t st =
          __hip_atomic_load(turn.wait_pair + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const uint64_t dt = wall_clock64() - t0;
      if (st >= 2 || dt >= kTurnWaitTicks || (st == 0 && dt >= kTurnStartTicks)) break;
      __builtin_amdgcn_s_sleep(8);
    }
  }
  // grid z: the target layers (one plan, each layer's own host records and cache)
  fetch_slice<U>(a, div_cpr, blockIdx.y, blockIdx.z,
                 blockIdx.x * (uint32_t)kFetchThreads + threadIdx.x,
                 gridDim.x * (uint32_t)kFetchThreads);
  if (turn.signal_pair && threadIdx.x == 0) {
    // this wave's host reads have all returned (its stores consumed them)
    const int32_t n = __hip_atomic_fetch_add(turn.signal_pair, 1, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT) + 1;
    if (n == turn.go)
      __hip_atomic_fetch_max(turn.signal_pair + 1, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__global__ void turns_reset_kernel(int32_t* turns, int32_t n) {
  for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    turns[i] = 0;
}

// Staged fetch: the records packed per unit in the device staging buffer go to their slots
// (16-byte pieces; grid y = unit). The staging layout and the plan range come from the host.
__global__ __launch_bounds__(256) void scatter_kernel(ScatterArgs a) {
  typedef unsigned int v4u __attribute__((ext_vector_type(4)));
  const int u = blockIdx.y;
  const int32_t* prefix = reinterpret_cast<const int32_t*>(a.stage);
  const int32_t first = prefix[u], n = prefix[u + 1] - first;
  const int32_t lo = (a.plan_count[u] * a.part_lo) >> 8;
  const uint32_t cpr = (uint32_t)a.R >> 4;
  const uint32_t total = (uint32_t)n * cpr;
  const uint8_t* src = a.stage + a.rec_offset + (int64_t)first * a.R;
  const int2* plan = a.plan + (int64_t)u * a.k + lo;
  uint8_t* cache = a.cache + (int64_t)u * a.B * a.R;
  for (uint32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < total;
       c += gridDim.x * blockDim.x) {
    const uint32_t r = c / cpr, w = c - r * cpr;
    const v4u v = *reinterpret_cast<const v4u*>(src + (int64_t)r * a.R + (w << 4));
    *reinterpret_cast<v4u*>(cache + (int64_t)plan[r].y * a.R + (w << 4)) = v;
  }
}

// Write-through (Section 3.3 (4)). One workgroup per (unit, share group). The table side is
// the canonical LRU applied to the one-position selection {pos}, specialised: the anchor's
// clock advances; a resident position has its stamp refreshed to 2t and its slot moved to the
// most-recent end of the recency index; a new position takes the least-recent slot order[0]
// (no slot is hit, so none is exempt) with the miss stamp 2t-1, and the index rotates by one.
// Then the unit's record of each of the group's layers is stored into that slot of the layer's
// cache and at pos in the layer's host pool. The index is staged in LDS for the shift.
__global__ __launch_bounds__(256) void admit_kernel(AdmitArgs a) {
  extern __shared__ uint16_t s_order[];  // [B] (slots < kMaxCapacity = 2^14)
  __shared__ int s_idx;
  typedef unsigned int v4u __attribute__((ext_vector_type(4)));
  const int unit = blockIdx.x, grp = blockIdx.y, tid = threadIdx.x, B = a.B;
  const int anchor = a.first + grp * a.G;
  const AnchorState st = a.states[anchor / a.G];
  const int32_t p = a.pos[unit];
  int32_t* slot_out = a.slots_out + (int64_t)grp * a.units + unit;
  if ((int64_t)p >= a.L) {  // invalid: latch the error, leave the unit's state untouched
    if (tid == 0) {
      *slot_out = -1;
      if (atomicCAS(&a.err[0], 0, (int)HISPARSE_ERR_BAD_SELECTION) == 0) {
        a.err[1] = anchor;
        a.err[2] = unit;
      }
      atomicAdd(&a.err[3], 1);
    }
    return;
  }
  const uint32_t t = st.clock[unit] + 1u;
  if (p < 0) {  // nothing to admit this event: only the clock advances
    if (tid == 0) {
      *slot_out = -1;
      st.clock[unit] = t;
    }
    return;
  }
  int32_t* pt = st.pt + (int64_t)unit * a.L;
  int32_t* slot_pos = st.slot_pos + (int64_t)unit * B;
  int32_t* order = st.order + (int64_t)unit * B;
  const int32_t hit = pt[p];
  if (tid == 0) s_idx = 0;  // stays in bounds even if the index were inconsistent
  __syncthreads();
  for (int j = tid; j < B; j += blockDim.x) {
    const int32_t s = order[j];
    s_order[j] = (uint16_t)s;
    if (s == hit) s_idx = j;  // the hit slot's place in the index (at most one thread)
  }
  __syncthreads();
  const int idx = hit >= 0 ? s_idx : 0;  // the entry that moves to the most-recent end
  const int32_t slot = (int32_t)s_order[idx];
  for (int j = idx + tid; j < B - 1; j += blockDim.x) order[j] = (int32_t)s_order[j + 1];
  if (tid == 0) {
    order[B - 1] = slot;
    if (hit >= 0) {
      st.slot_ts[(int64_t)unit * B + slot] = 2u * t;
    } else {
      const int32_t old = slot_pos[slot];
      if (old >= 0) pt[old] = -1;  // the evicted record becomes host-only
      pt[p] = slot;
      slot_pos[slot] = p;
      st.slot_ts[(int64_t)unit * B + slot] = 2u * t - 1u;
    }
    *slot_out = slot;
    st.clock[unit] = t;
  }
  if (!a.write) return;
  const int z_end = min(anchor + a.G, a.first + a.n_layers);
  for (int z = anchor; z < z_end; ++z) {
    const uint8_t* src = a.records + ((int64_t)(z - a.first) * a.units + unit) * a.R;
    uint8_t* cache = a.layers[z].cache + ((int64_t)unit * B + slot) * a.R;
    uint8_t* host = a.layers[z].host + ((int64_t)unit * a.L + p) * a.R;
    for (int q = tid; q < (a.R >> 4); q += blockDim.x) {
      const v4u v = *reinterpret_cast<const v4u*>(src + 16 * q);
      *reinterpret_cast<v4u*>(cache + 16 * q) = v;
      *reinterpret_cast<v4u*>(host + 16 * q) = v;
    }
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
hipError_t launch_resolve_nt(const ResolveArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(resolve_kernel<NT>, dim3(a.units), dim3(NT), resolve_lds_bytes(a.k, a.B),
                     stream, a);
  return hipGetLastError();
}

}  // namespace

size_t resolve_lds_bytes(int32_t k, int32_t B) {
  const size_t k4 = (size_t)((k + 3) & ~3);
  return 16 * k4 + 8 * (size_t)((B + 31) >> 5) + 4 * (size_t)kBuckets;
}

int resolve_threads(int32_t B) {
  int nt = 64;
  while (nt < 1024 && nt * kMaxChunk < B) nt <<= 1;
  while (nt < 1024 && nt * 4 < B) nt <<= 1;  // about four order entries per thread
  return nt;
}

hipError_t launch_resolve(const ResolveArgs& a, hipStream_t stream) {
  const int nt = resolve_threads(a.B);
  if (a.k > kMaxPer * nt) return hipErrorInvalidValue;  // excluded by descriptor validation
  switch (nt) {
    case 64: return launch_resolve_nt<64>(a, stream);
    case 128: return launch_resolve_nt<128>(a, stream);
    case 256: return launch_resolve_nt<256>(a, stream);
    case 512: return launch_resolve_nt<512>(a, stream);
    default: return launch_resolve_nt<1024>(a, stream);
  }
}

hipError_t read_resolve_phase_stamps(uint64_t* host, int32_t units) {
#ifdef HISPARSE_PHASE_STAMPS
  return hipMemcpyFromSymbol(host, HIP_SYMBOL(g_phase_stamps),
                             (size_t)units * kPhaseStamps * sizeof(uint64_t), 0,
                             hipMemcpyDeviceToHost);
#else
  (void)host;
  (void)units;
  return hipErrorNotSupported;
#endif
}

hipError_t launch_scatter(const ScatterArgs& a, hipStream_t stream) {
  // a few workgroups per unit: each unit's run is at most k records (HBM to HBM)
  const int per_unit = std::max(1, std::min(64, 256 / std::max(1, a.units)));
  hipLaunchKernelGGL(scatter_kernel, dim3(per_unit, a.units), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_fetch(const FetchArgs& a, int transfer_block_bytes, int workgroups,
                        hipStream_t stream, const LinkTurn* turn) {
  const int U = transfer_block_bytes / 16;
  const int64_t max_chunks = (int64_t)a.k * (a.R / 16);
  int64_t x = (max_chunks + (int64_t)kFetchThreads * U - 1) / ((int64_t)kFetchThreads * U);
  // the workgroup budget is shared by the launch's (unit, layer) pairs; each pair's workgroups
  // stride over its plan, so any x >= 1 covers it
  const int64_t cap = std::max<int64_t>(1, workgroups / ((int64_t)a.units * a.n_layers));
  if (x > cap) x = cap;
  const dim3 grid((unsigned)x, (unsigned)a.units, (unsigned)a.n_layers);
  const FastDiv f = make_fastdiv((uint32_t)(a.R / 16));
  TurnDev t{nullptr, nullptr, 0};
  if (turn && turn->turns) {
    const int64_t wgs = x * a.units * a.n_layers;
    if (turn->wait >= 0) t.wait_pair = turn->turns + 2 * (int64_t)turn->wait;
    if (turn->signal >= 0) t.signal_pair = turn->turns + 2 * (int64_t)turn->signal;
    t.go = (int32_t)std::max<int64_t>(1, (wgs * turn->share + 255) / 256);
  }
  switch (U) {
    case 1: hipLaunchKernelGGL(fetch_kernel<1>, grid, dim3(kFetchThreads), 0, stream, a, f, t); break;
    case 2: hipLaunchKernelGGL(fetch_kernel<2>, grid, dim3(kFetchThreads), 0, stream, a, f, t); break;
    case 4: hipLaunchKernelGGL(fetch_kernel<4>, grid, dim3(kFetchThreads), 0, stream, a, f, t); break;
    case 8: hipLaunchKernelGGL(fetch_kernel<8>, grid, dim3(kFetchThreads), 0, stream, a, f, t); break;
    default: hipLaunchKernelGGL(fetch_kernel<16>, grid, dim3(kFetchThreads), 0, stream, a, f, t); break;
  }
  return hipGetLastError();
}

hipError_t launch_turns_reset(int32_t* turns, int32_t n_turns, hipStream_t stream) {
  const int32_t n = 2 * n_turns;
  const int blocks = std::max(1, std::min(64, (n + 255) / 256));
  hipLaunchKernelGGL(turns_reset_kernel, dim3(blocks), dim3(256), 0, stream, turns, n);
  return hipGetLastError();
}

hipError_t launch_admit(const AdmitArgs& a, int32_t n_groups, hipStream_t stream) {
  static_assert(kMaxCapacity <= 65536, "16-bit slots in the admission kernel's LDS");
  hipLaunchKernelGGL(admit_kernel, dim3(a.units, n_groups), dim3(256), (size_t)a.B * 2, stream,
                     a);
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
