// Sparse decode attention over gathered records for gfx950 (the consumer of the resolve
// step's slot vector, Section 3.4 Phase 5; exactness per Section 3.1).
//
// For each unit and query head h:  out_h = sum_j softmax_j(scale * q_h . key_j) value_j,
// over the tokens of the k selected records, in the order of the slot vector.
//
// Structure (every attention kernel: one workgroup per (unit, token split, head block); each
// 32-token chunk is staged into LDS once with direct global->LDS loads and shared by the
// workgroup's head waves)
//   attn_partial_kernel  grouped-query records (d 128). A wave owns 16 query heads (the MFMA N
//     dimension) and one 32-token chunk per iteration.
//       S^T[token][head] = K[token][:] . Q^T[:][head]     v_mfma_f32_16x16x32_bf16, K from LDS
//                                                        rows, Q resident in VGPRs
//       online softmax in fp32 (exp2, reference max per head), P rounded to bf16
//       O[head][dim]   += P[head][token] . V[token][dim]  v_mfma_f32_16x16x32_bf16, V by LDS
//                                                        transpose reads
//     A lane's S^T accumulator holds tokens {4g..4g+3, 16+4g..16+4g+3} (g = lane/16) of its
//     head, which is exactly one P operand when the PV contraction index runs over the tokens
//     in that order, so P never leaves the lane; the V operand is read in the same order.
//   attn_mla_kernel  latent records (d_qk 576, d_v 512 = the key's first 512 dims): 32 heads
//     per wave on v_mfma_f32_32x32x16_bf16, the output in accumulation registers.
//   attn_combine_kernel / attn_combine_mla_kernel  merge the per-split (max, sum, unnormalised
//     output) triples of each (unit, head) in ascending split order.
//   Either attention kernel can carry an exact-prefetch replay: extra workgroups after the
//   attention's copy records into other layers' caches and exit (replay_worker).
// The reduction order depends only on token positions in the sequence, never on the slot
// values, so any placement of the same records gives bit-identical outputs.
#include <math.h>

#include <algorithm>

#include "fetch_device.h"

namespace hisparse {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChunk = 32;            // tokens per wave per iteration
constexpr int kTargetWorkgroups = 256;
constexpr int kMaxSplitRecords = 1024;  // record indices of one split staged in LDS
// Rescale the running output only when a head's running max grows by more than this (log2
// units): exponentials are taken against a slightly stale max (values up to 2^8), which is
// exact softmax arithmetic with a different reference point and keeps fp32/bf16 far from
// overflow; the final normalisation uses the same reference.
constexpr float kRescaleSlack = 8.0f;

// 16-byte loads of padding tokens and padding slots read zeros from here.
__device__ __attribute__((aligned(16))) uint8_t g_zero_token[2048];

// A replay carried by a launch (attention or merge): the extra workgroups after the launch's
// own, per_pair of them for each (unit, target layer) of the plan.
struct CarriedReplay {
  FetchArgs pf;
  FastDiv pf_div;
  int32_t pf_per_pair, pf_wg, pf_u;  // pf_u: 16-byte loads each replay thread keeps in flight
};

struct AttnArgs {
  const uint8_t* pool;
  const uint16_t* q;
  const int32_t* idx;
  float* part_o;    // [units][n_parts][H][DV]
  float2* part_ml;  // [units][n_parts][H] (running max in log2 units, running sum)
  int64_t rec_per_unit;
  int32_t R, token_bytes, tpr_shift, k, H, n_tok;
  int32_t split_tokens, n_wg_splits, hb, n_parts, n_wg;
  int32_t Hp;         // latent attention: heads rounded up to 32 (partial-output block layout)
  int32_t idx_units;  // unit u reads index row u % idx_units
  float scale_log2;
  // A prefetch replay carried by the launch: extra workgroups after the attention workgroups
  // copy that plan's records (pf_wg = 0: none).
  CarriedReplay rp;
};

// Extra workgroup e of a launch: its share of the carried replay. It shares no memory with the
// launch's own workgroups (other layers' caches), so it needs no synchronisation.
__device__ __forceinline__ void replay_worker(const CarriedReplay& r, int e) {
  const int pair = e / r.pf_per_pair, x = e - pair * r.pf_per_pair;
  const int unit = pair % r.pf.units, z = pair / r.pf.units;
  const uint32_t first = x * blockDim.x + threadIdx.x, stride = r.pf_per_pair * blockDim.x;
  if (r.pf_u >= 4) fetch_slice<4>(r.pf, r.pf_div, unit, z, first, stride);
  else if (r.pf_u == 2) fetch_slice<2>(r.pf, r.pf_div, unit, z, first, stride);
  else fetch_slice<1>(r.pf, r.pf_div, unit, z, first, stride);
}

// Latent-attention partial outputs are stored in the PV accumulators' own layout, so every
// lane writes 16 contiguous bytes: per part, 32-head block b, output tile n (dims 32n..32n+31),
// group q and lane L hold heads 32b + 8q + 4(L >> 5) + e, e = 0..3, of dim 32n + (L & 31).
__device__ __host__ inline int64_t mla_part_offset(int head, int dim) {
  const int hl = head & 31, q = hl >> 3, e = hl & 3, ln = ((hl >> 2) & 1) * 32 + (dim & 31);
  return (int64_t)(head >> 5) * 32 * 512 + ((((dim >> 5) * 4 + q) * 64 + ln) * 4 + e);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two softmax weights 2^(s0 - m), 2^(s1 - m) rounded to bf16 (nearest even, one packed
// v_cvt_pk_bf16_f32), the first in the low half; *psum accumulates the rounded values in that
// order. The exponential is the hardware v_exp_f32: weights below 2^-126 flush to zero.
__device__ inline uint32_t weights_bf16x2(float s0, float s1, float m, float* psum) {
  const f32x2 e = {__builtin_amdgcn_exp2f(s0 - m), __builtin_amdgcn_exp2f(s1 - m)};
  const uint32_t w = __builtin_bit_cast(uint32_t, __builtin_convertvector(e, bf16x2_t));
  *psum += __uint_as_float(w << 16);
  *psum += __uint_as_float(w & 0xFFFF0000u);
  return w;
}
__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }


typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) void lds_void;

// LDS reads that the compiler does not see as memory accesses. In the latent-attention loop the
// next chunk's direct-to-LDS loads are in flight while the current chunk is read from another
// buffer; before a compiler-visible LDS read the compiler would wait for those loads (it cannot
// tell the buffers apart), which takes the load of chunk it+1 out from under the compute of
// chunk it. The caller waits for these reads itself, with s_waitcnt lgkmcnt(N), N = the number
// of its own reads issued after the one it needs: LDS reads complete in order, so any other
// LGKM operation in flight can only lengthen that wait.
__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const lds_void*)p;
}
__device__ inline u32x4 lds_read_b128(uint32_t addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}
__device__ inline v4i16 lds_read_tr16_b64(uint32_t addr) {
  v4i16 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}
// Wait until at most N LGKM operations are outstanding; a and b are the registers of the reads
// waited for (tied, so that their users stay after the wait).
template <int N>
__device__ __forceinline__ void lgkm_wait2(v4i16& a, v4i16& b) {
  asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "n"(N));
}
// The same for two 16-byte reads, with n (a constant once the caller's loop is unrolled, at
// most M) selecting the count.
template <int M>
__device__ __forceinline__ void lgkm_wait2_upto(int n, u32x4& a, u32x4& b) {
  if constexpr (M >= 0) {
    if (n == M) asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "n"(M));
    else lgkm_wait2_upto<M - 1>(n, a, b);
  }
}
// S^T += K . Q^T for one k-step once the K rows' read (with at most N later LDS reads) is in;
// the first step of a chain (FIRST) starts from zero. The s_nop covers the wait states after a
// just-written operand that the compiler does not see through the assembly.
template <int N, bool FIRST>
__device__ __forceinline__ void mfma_qk(f32x16& acc, const u32x4& k, const bf16x8_t& q) {
  if constexpr (FIRST)
    asm volatile("s_waitcnt lgkmcnt(%3)\n\ts_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, 0"
                 : "=&v"(acc) : "v"(k), "v"(q), "n"(N));
  else
    asm volatile("s_waitcnt lgkmcnt(%3)\n\ts_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0"
                 : "+v"(acc) : "v"(k), "v"(q), "n"(N));
}

// Wait until at most N direct-to-LDS loads of this wave are outstanding and its LDS writes are
// done, then synchronise the workgroup. (A workgroup fence would also drain the younger
// prefetches, which is exactly what the pipeline must not do.)
template <int N>
__device__ inline void wait_loads_and_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// LDS tile of one 32-token chunk: token t's 16-byte piece c at slot t * PP + c, PP >= P pieces
// per row. The padding makes consecutive rows start 36 (MLA: PP = 73) or 20 (GQA: PP = 37)
// banks apart, so the 16 rows read by one MFMA operand load hit distinct banks, and the
// transpose reads (4 rows x 4 column pairs per 16 lanes) do too.
template <int P>
struct TileRow {
  static constexpr int PP = (P == 72) ? 73 : (P == 32 ? 37 : P + 1);
};

// Row order of a 32-token chunk inside the MFMA tiles: operand row m of tile h reads token
// 16h + perm(m) with perm(4g + s) = 8 (g >> 1) + 2s + (g & 1). A lane's S^T accumulator then
// holds tokens perm(4g + j) (+16), and the PV transpose reads touch rows two apart, which
// with the padded row stride keeps both access patterns free of bank conflicts.
__device__ inline int tile_row(int m) { return 8 * (m >> 3) + 2 * (m & 3) + ((m >> 2) & 1); }

// Direct global->LDS staging of one 32-token chunk starting at token cbase into `tile`.
// Lane t < kChunk first resolves token t of the chunk to its byte offset in the unit's pool
// (-1: padding token, padding slot or past the split end; such rows read zeros, and their
// scores are masked to -inf so they carry P = 0). Load j (64 lanes) fills tile slots
// 64j .. 64j+63, which span at most three tile rows: each lane takes its row's offset from the
// lane that resolved it (scalar lane reads) and adds its 16-byte piece. The calling wave
// issues loads [j0, j0 + n_loads) of the chunk.
template <int P, int PP, int LPW_MAX>
__device__ __forceinline__ void stage_chunk(uint16_t* tile, const int32_t* s_idx,
                                            const uint8_t* pool_u, int cbase, int tok_end,
                                            int rec_begin, int tpr_shift, int R, int token_bytes,
                                            int j0, int n_loads) {
  // recompute the per-lane arithmetic here instead of keeping it live across the loop
  int lane = threadIdx.x & 63;
  asm volatile("" : "+v"(lane));
  const int tk = cbase + lane;
  const bool in_chunk = lane < kChunk && tk < tok_end;
  const int32_t s = s_idx[in_chunk ? (tk >> tpr_shift) - rec_begin : 0];
  const int toff =
      (in_chunk && s >= 0) ? s * R + (tk & ((1 << tpr_shift) - 1)) * token_bytes : -1;
#pragma unroll
  for (int jj = 0; jj < LPW_MAX; ++jj) {
    if (jj < n_loads) {  // wave-uniform
      const int j = j0 + jj;
      const int t0 = (64 * j) / PP;
      int c = 64 * j - t0 * PP + lane;
      int o = __builtin_amdgcn_readlane(toff, t0);
      const int o1 = __builtin_amdgcn_readlane(toff, t0 + 1);
      if (c >= PP) { c -= PP; o = o1; }
      if constexpr (PP < 64) {  // a load of 64 slots can reach a third row
        const int o2 = __builtin_amdgcn_readlane(toff, t0 + 2);
        if (c >= PP) { c -= PP; o = o2; }
      }
      const bool real = o >= 0 && c < P;
      const uint8_t* src =
          real ? pool_u + (uint32_t)o + 16 * c : g_zero_token + 16 * (c < P ? c : 0);
      __builtin_amdgcn_global_load_lds(src, (lds_void*)(tile + 64 * j * 8), 16, 0, 0);
    }
  }
}

// The calling wave's loads of the current chunk are done once at most `younger` later chunks'
// loads (n_loads each) are outstanding; then the workgroup synchronises.
template <int NST, int LPW_MAX, int LPW_MIN>
__device__ __forceinline__ void wait_chunk(int younger, bool max_loads) {
  if constexpr (NST == 2) {
    wait_loads_and_barrier<0>();
  } else if (max_loads) {
    if (younger >= 2) wait_loads_and_barrier<(NST - 2) * LPW_MAX>();
    else if (younger == 1) wait_loads_and_barrier<LPW_MAX>();
    else wait_loads_and_barrier<0>();
  } else {
    if (younger >= 2) wait_loads_and_barrier<(NST - 2) * LPW_MIN>();
    else if (younger == 1) wait_loads_and_barrier<LPW_MIN>();
    else wait_loads_and_barrier<0>();
  }
}

template <int DQK, int DV, int VOFF, int HW, int TW, int NST>
__global__ __launch_bounds__(64 * HW * TW, (HW * TW >= 8) ? 2 : 1)
void attn_partial_kernel(AttnArgs a) {
  constexpr int TE = (DQK > VOFF + DV) ? DQK : VOFF + DV;  // bf16 per token used here
  constexpr int P = TE / 8;                                 // 16-byte pieces per token
  constexpr int PP = TileRow<P>::PP;                        // pieces per LDS row
  constexpr int NL = ((kChunk - 1) * PP + P + 63) / 64;     // 64-lane loads per chunk
  constexpr int TILE = NL * 64 * 8;                         // bf16 per chunk tile
  constexpr int LPW_MAX = (NL + HW - 1) / HW;               // loads per wave (first waves)
  constexpr int LPW_MIN = NL / HW;                          // loads per wave (last waves)
  constexpr int NL_REM = NL % HW;                           // waves doing LPW_MAX loads
  constexpr int NKK = DQK / 32;
  constexpr int NOUT = DV / 16;
  static_assert(DQK % 32 == 0 && DV % 16 == 0 && VOFF % 8 == 0, "shape");
  static_assert(NST >= 2 && NST <= 4 && (NST - 2) * LPW_MAX < 64, "pipeline depth");
  __shared__ __align__(16) uint16_t s_kv[TW * NST * TILE];
  __shared__ int32_t s_idx[kMaxSplitRecords];  // the split's record indices, -1 = skip
  __shared__ uint32_t s_valid[kMaxSplitTokens / 32];  // bit t of word c: token 32c+t attends

  // XCD-aware mapping: consecutive workgroup ids go round-robin over the 8 XCDs, so give each
  // XCD a contiguous range of work items; the head blocks of one (unit, split) then share the
  // staged records through the same L2.
  const int nwg_pad = (a.n_wg + 7) & ~7;
  if ((int)blockIdx.x >= nwg_pad) {  // wave-uniform: the whole workgroup replays
    replay_worker(a.rp, (int)blockIdx.x - nwg_pad);
    return;
  }
  const int w = (int)(blockIdx.x & 7) * (nwg_pad >> 3) + (int)(blockIdx.x >> 3);
  if (w >= a.n_wg) return;
  const int hb = w % a.hb;
  const int split = (w / a.hb) % a.n_wg_splits;
  const int unit = w / (a.hb * a.n_wg_splits);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hg = wave % HW, tg = wave / HW;
  const int g = lane >> 4;
  uint16_t* s_tiles = s_kv + tg * NST * TILE;

  const int tok_begin = split * a.split_tokens;
  const int tok_end = min(a.n_tok, tok_begin + a.split_tokens);
  const int rec_begin = tok_begin >> a.tpr_shift;
  const int n_rec = ((tok_end - 1) >> a.tpr_shift) - rec_begin + 1;
  {
    const int32_t* idx_u = a.idx + (int64_t)(unit % a.idx_units) * a.k + rec_begin;
    for (int i = tid; i < n_rec; i += 64 * HW * TW) {
      const int32_t s = idx_u[i];
      s_idx[i] = (s >= 0 && s < a.rec_per_unit) ? s : -1;
    }
  }
  const uint8_t* pool_u = a.pool + (int64_t)unit * a.rec_per_unit * a.R;

  const int head = hb * 16 * HW + hg * 16 + (lane & 15);
  const bool head_ok = head < a.H;

  f32x4 o[NOUT];
#pragma unroll
  for (int n = 0; n < NOUT; ++n) o[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  __syncthreads();  // s_idx is ready
  // Q^T operand, loaded unconditionally (a head past H reads head 0's row: its scores are never
  // stored and, being head 0's, move no reference max that head 0 does not) and before the
  // validity masks are written and the first chunks issued, so that it is in flight meanwhile
  bf16x8_t qreg[NKK];
  {
    const uint16_t* qrow = a.q + ((int64_t)unit * a.H + (head_ok ? head : 0)) * DQK + 8 * g;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      qreg[kk] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(qrow + kk * 32));
  }
  const int n_it = (tok_end - tok_begin + kChunk * TW - 1) / (kChunk * TW);
  {
    // every chunk the token groups iterate over gets its word, including chunks that lie
    // wholly past the split end (all zero)
    const int span = n_it * kChunk * TW;
    for (int base = wave * 64; base < span; base += 64 * HW * TW) {
      const int tk = tok_begin + base + lane;
      const bool ok = tk < tok_end && s_idx[(tk >> a.tpr_shift) - rec_begin] >= 0;
      const uint64_t m = __ballot(ok);
      if (lane == 0) {
        s_valid[base >> 5] = (uint32_t)m;
        if (base + 32 < span) s_valid[(base >> 5) + 1] = (uint32_t)(m >> 32);
      }
    }
  }

  // wave hg stages loads [j0, j0 + n_loads) of each chunk of its token group
  const int hg_s = __builtin_amdgcn_readfirstlane(hg);
  const int n_loads = hg_s < NL_REM ? LPW_MAX : LPW_MIN;
  const int j0 = hg_s * LPW_MIN + min(hg_s, NL_REM);
  auto issue = [&](int it, int buf) {
    stage_chunk<P, PP, LPW_MAX>(s_tiles + buf * TILE, s_idx, pool_u,
                                tok_begin + it * kChunk * TW + tg * kChunk, tok_end, rec_begin,
                                a.tpr_shift, a.R, a.token_bytes, j0, n_loads);
  };
  auto wait = [&](int younger) { wait_chunk<NST, LPW_MAX, LPW_MIN>(younger, hg < NL_REM); };

#pragma unroll
  for (int st = 0; st < NST - 1; ++st)
    if (st < n_it) issue(st, st);

  // Per chunk: scores (QK), softmax against the running reference max, then P.V. O is touched
  // only by MFMAs inside the loop; the rare move of a head's reference max (growth beyond the
  // slack) leaves the loop, rescales, finishes that chunk and re-enters.
  f32x4 s0, s1;
  float sc[8];
  float cmax = -INFINITY;
  int it = 0;

  auto finish_chunk = [&](const uint16_t* tile) {
    uint32_t pw[4];
    float psum = 0.f;
    if (m_run == -INFINITY) {
      pw[0] = pw[1] = pw[2] = pw[3] = 0u;
    } else {
#pragma unroll
      for (int j = 0; j < 8; j += 2) pw[j >> 1] = weights_bf16x2(sc[j], sc[j + 1], m_run, &psum);
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run += psum;
    const bf16x8_t pa = __builtin_bit_cast(bf16x8_t, u32x4{pw[0], pw[1], pw[2], pw[3]});
    // V operand by transpose reads: in each 16-lane group, lane 4s+q addresses
    // V[token][16n + 4q .. +3] of token perm(4g+s) (first read) or 16+perm(4g+s) (second
    // read); lane t then holds V[those tokens][16n + t], i.e. B[k = 8g .. 8g+7][n = t], in the
    // token order of this lane's P values.
    const int ts = (lane & 15) >> 2, q4 = (lane & 3) * 4;
    const uint32_t vrow0 = lds_addr(tile + tile_row(4 * g + ts) * PP * 8 + VOFF + q4);
    const uint32_t vrow1 = vrow0 + 2 * (16 * PP * 8);
    // transpose reads VD output tiles ahead of their MFMAs (opaque LDS reads, see lds_read_b128)
    constexpr int VD = 3;
    static_assert(VD == 3 && NOUT > VD, "the waits below count a ring of 3 read pairs");
    v4i16 vlo[VD], vhi[VD];
    auto vread = [&](int n, int slot) {
      vlo[slot] = lds_read_tr16_b64(vrow0 + 2 * 16 * n);
      vhi[slot] = lds_read_tr16_b64(vrow1 + 2 * 16 * n);
    };
#pragma unroll
    for (int n = 0; n < VD; ++n) vread(n, n);
#pragma unroll
    for (int n = 0; n < NOUT; ++n) {
      // the reads issued after tile n's pair: those of tiles n+1 .. min(n+VD-1, NOUT-1)
      const int later = NOUT - 1 - n < VD - 1 ? NOUT - 1 - n : VD - 1;
      if (later == 2) lgkm_wait2<4>(vlo[n % VD], vhi[n % VD]);
      else if (later == 1) lgkm_wait2<2>(vlo[n % VD], vhi[n % VD]);
      else lgkm_wait2<0>(vlo[n % VD], vhi[n % VD]);
      const bf16x8_t vb = __builtin_bit_cast(
          bf16x8_t, __builtin_shufflevector(vlo[n % VD], vhi[n % VD], 0, 1, 2, 3, 4, 5, 6, 7));
      o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vb, o[n], 0, 0, 0);
      if (n + VD < NOUT) vread(n + VD, n % VD);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  for (;;) {
    for (; it < n_it; ++it) {
      // chunks it+1 .. it+NST-2 were issued earlier and may still be in flight
      wait(min(NST - 2, n_it - 1 - it));
      const uint16_t* tile = s_tiles + (it % NST) * TILE;
      const int cbase = tok_begin + it * kChunk * TW + tg * kChunk;
      // the chunk's validity word, read before the next chunk's loads are issued
      const uint32_t vmask = s_valid[(cbase - tok_begin) >> 5];
      __builtin_amdgcn_sched_barrier(0);
      // every wave is past its reads of buffer (it-1) % NST: refill it with chunk it+NST-1
      if (it + NST - 1 < n_it) issue(it + NST - 1, (it + NST - 1) % NST);

      // ---- scores: S^T tiles for tokens [0,16) and [16,32) of the chunk ----
      // all K reads first (opaque LDS reads, see lds_read_b128), then each k-step's MFMAs once
      // its pair is in
      s0 = f32x4{0.f, 0.f, 0.f, 0.f};
      s1 = f32x4{0.f, 0.f, 0.f, 0.f};
      const uint32_t k0 = lds_addr(tile + (tile_row(lane & 15) * PP + g) * 8);
      const uint32_t k1 = k0 + 2 * (16 * PP * 8);
      static_assert(NKK <= 8, "lgkmcnt holds at most 15 outstanding reads");
      u32x4 ka[NKK], kb[NKK];
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        ka[kk] = lds_read_b128(k0 + 2 * kk * 32);
        kb[kk] = lds_read_b128(k1 + 2 * kk * 32);
      }
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        lgkm_wait2_upto<2 * (NKK - 1)>(2 * (NKK - 1 - kk), ka[kk], kb[kk]);
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ka[kk]),
                                                    qreg[kk], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kb[kk]),
                                                    qreg[kk], s1, 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      int gq = g;
      asm volatile("" : "+v"(gq));
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int bit = j < 4 ? tile_row(4 * gq + j) : 16 + tile_row(4 * gq + (j - 4));
        const float raw = j < 4 ? s0[j] : s1[j - 4];
        sc[j] = ((vmask >> bit) & 1u) ? raw * a.scale_log2 : -INFINITY;
      }
      cmax = sc[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) cmax = fmaxf(cmax, sc[j]);
      cmax = fmaxf(cmax, __shfl_xor(cmax, 16, 64));
      cmax = fmaxf(cmax, __shfl_xor(cmax, 32, 64));
      // Validity is per token, so every head of the wave agrees on whether m_run is -inf.
      // While it is, O and l are exactly zero and the reference max can simply be set.
      if (m_run == -INFINITY) m_run = cmax;
      else if (__ballot(cmax > m_run + kRescaleSlack)) break;
      finish_chunk(tile);
    }
    if (it >= n_it) break;
    // rare path: move the reference max of the heads whose scores outgrew it
    const float m_new = fmaxf(m_run, cmax);
    const float alpha = exp2f(m_run - m_new);
    l_run *= alpha;
    m_run = m_new;
    float al[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) al[j] = __shfl(alpha, 4 * g + j, 64);
#pragma unroll
    for (int n = 0; n < NOUT; ++n) {
#pragma unroll
      for (int j = 0; j < 4; ++j) o[n][j] *= al[j];
    }
    finish_chunk(s_tiles + (it % NST) * TILE);
    ++it;
  }

  // ---- partial results of this (split, token group) ----
  const int part = split * TW + tg;
  float* po = a.part_o + ((int64_t)unit * a.n_parts + part) * a.H * DV;
  const int head_base = hb * 16 * HW + hg * 16 + 4 * g;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int h = head_base + j;
    if (h < a.H) {
#pragma unroll
      for (int n = 0; n < NOUT; ++n) po[(int64_t)h * DV + n * 16 + (lane & 15)] = o[n][j];
    }
  }
  if (lane < 16 && head_ok)
    a.part_ml[((int64_t)unit * a.n_parts + part) * a.H + head] = make_float2(m_run, l_run);
}

// Logical row r of a 32-token MFMA tile -> LDS tile row (token) for the latent-attention kernel.
// With r = 16a + 8b + 4h + s the row is 16a + 4s + 2b + h: the P operand of a lane (k-step a,
// half h) then comes straight from its S^T accumulator, and each group of 16 lanes of a V
// transpose read touches rows 4 apart, i.e. four row bases 16 banks apart under the padded
// stride, so those reads are free of bank conflicts; the 16 K rows one operand load reads are
// a permutation of 16 consecutive rows, which are conflict-free as well.
__device__ inline int mla_row(int r) {
  return 16 * (r >> 4) + 4 * (r & 3) + 2 * ((r >> 3) & 1) + ((r >> 2) & 1);
}

// Scores of the latent-attention kernel may exceed the split's reference by this many powers
// of two: P <= 2^64 and sums over at most 8192 tokens stay far inside the fp32/bf16 range.
constexpr float kMlaSlack = 64.0f;

// Exact fallback for a latent-attention split whose scores outgrow the reference: plain online
// softmax with fp32 rescaling, one head at a time per wave, K and V read straight from the
// pool. Writes the split's partial results in the fast path's format. Only inputs whose scores
// span more than kMlaSlack powers of two within one split ever come here.
__device__ __forceinline__ void mla_split_exact(const AttnArgs& a, const int32_t* s_idx,
                                                const uint32_t* s_valid, int unit, int split,
                                                int tok_begin, int tok_end, int rec_begin,
                                                int head0) {
  constexpr int DQK = 576, DV = 512;
  const int lane = threadIdx.x & 63;
  const uint8_t* pool_u = a.pool + (int64_t)unit * a.rec_per_unit * a.R;
  const int tpr_mask = (1 << a.tpr_shift) - 1;
  for (int hh = 0; hh < 32; ++hh) {
    const int head = head0 + hh;
    if (head >= a.H) break;
    const uint16_t* qh = a.q + ((int64_t)unit * a.H + head) * DQK;
    float qv[DQK / 64];
#pragma unroll
    for (int i = 0; i < DQK / 64; ++i) qv[i] = bf16_to_f32(qh[lane + 64 * i]);
    float m = -INFINITY, l = 0.f, acc[DV / 64];
#pragma unroll
    for (int e = 0; e < DV / 64; ++e) acc[e] = 0.f;
    for (int t = tok_begin; t < tok_end; ++t) {
      const int bit = t - tok_begin;
      if (!((s_valid[bit >> 5] >> (bit & 31)) & 1u)) continue;
      const int rec = s_idx[(t >> a.tpr_shift) - rec_begin];
      const uint16_t* kt = reinterpret_cast<const uint16_t*>(
          pool_u + (int64_t)rec * a.R + (int64_t)(t & tpr_mask) * a.token_bytes);
      float d = 0.f;
#pragma unroll
      for (int i = 0; i < DQK / 64; ++i) d += qv[i] * bf16_to_f32(kt[lane + 64 * i]);
#pragma unroll
      for (int x = 32; x >= 1; x >>= 1) d += __shfl_xor(d, x, 64);
      const float sc = d * a.scale_log2;
      const float m_new = fmaxf(m, sc);
      const float alpha = exp2f(m - m_new);
      const float pr = exp2f(sc - m_new);
      l = l * alpha + pr;
#pragma unroll
      for (int e = 0; e < DV / 64; ++e)
        acc[e] = acc[e] * alpha + pr * bf16_to_f32(kt[lane * (DV / 64) + e]);
      m = m_new;
    }
    float* po = a.part_o + ((int64_t)unit * a.n_parts + split) * a.Hp * DV;
#pragma unroll
    for (int e = 0; e < DV / 64; ++e) po[mla_part_offset(head, lane * (DV / 64) + e)] = acc[e];
    if (lane == 0)
      a.part_ml[((int64_t)unit * a.n_parts + split) * a.H + head] = make_float2(m, l);
  }
}

// Latent attention (d_qk 576, d_v 512 = the first 512 key dims). One workgroup per
// (unit, token split, head block of 32 * HW heads); wave w owns 32 heads (w % HW) of token
// group w / HW. Each token group has its own ring of NST chunk tiles in LDS, staged once for its
// HW head waves; with TG = 2 groups the split's 32-token chunks alternate between the groups and
// the two groups' results are merged in LDS at the end, so a workgroup writes one partial result
// for twice the tokens of one group (half the partial traffic of two workgroups).
//   S^T[token][head] = K[token][:] . Q^T[:][head]   v_mfma_f32_32x32x16_bf16, 36 k-steps, K rows
//                                                   from LDS, Q resident in VGPRs
//   O[head][dim]    += P[head][token] . V[token][dim]  v_mfma_f32_32x32x16_bf16, 2 k-steps x 16
//                                                   output tiles, V by LDS transpose reads
// A lane holds 16 of a head's 32 scores (the other 16 are in lane ^ 32), which are exactly its
// P operands of the two PV k-steps; O (16 tiles x 16 fp32 per lane) lives in accumulators.
template <int HW, int TG, int NST, bool PACED>
__global__ __launch_bounds__(64 * HW * TG, 1)
void attn_mla_kernel(AttnArgs a) {
  constexpr int DQK = 576, DV = 512;
  constexpr int NW = HW * TG;
  constexpr int P = DQK / 8;                              // 16-byte pieces per token
  constexpr int PP = TileRow<P>::PP;                      // pieces per LDS row
  constexpr int NL = ((kChunk - 1) * PP + P + 63) / 64;   // 64-lane loads per chunk
  constexpr int TILE = NL * 64 * 8;                       // bf16 per chunk tile
  constexpr int LPW_MAX = (NL + HW - 1) / HW;             // a group's loads per head wave
  constexpr int LPW_MIN = NL / HW;
  constexpr int NL_REM = NL % HW;
  constexpr int NKK = DQK / 16;  // QK k-steps
  constexpr int NDV = DV / 32;   // PV output tiles
  static_assert(NST >= 2 && NST <= 4 && (NST - 2) * LPW_MAX < 64, "pipeline depth");
  static_assert(TG == 1 || TG == 2, "token groups");
  static_assert(TG == 1 || TG * NST * TILE * 2 >= HW * (64 * 64 * 16 + 32 * 8),
                "the tiles hold one group's results for the merge");
  __shared__ __align__(16) uint16_t s_kv[TG * NST * TILE];
  __shared__ int32_t s_idx[kMaxSplitRecords];         // the split's record indices, -1 = skip
  __shared__ uint32_t s_valid[kMaxSplitTokens / 32];  // bit t of word c: token 32c+t attends
  __shared__ int s_fallback;                           // some score outgrew its reference

  // XCD-aware mapping, as in attn_partial_kernel
  const int nwg_pad = (a.n_wg + 7) & ~7;
  if ((int)blockIdx.x >= nwg_pad) {  // wave-uniform: the whole workgroup replays
    replay_worker(a.rp, (int)blockIdx.x - nwg_pad);
    return;
  }
  const int w = (int)(blockIdx.x & 7) * (nwg_pad >> 3) + (int)(blockIdx.x >> 3);
  if (w >= a.n_wg) return;
  const int hb = w % a.hb;
  const int split = (w / a.hb) % a.n_wg_splits;
  const int unit = w / (a.hb * a.n_wg_splits);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int hg = wave % HW, tg = wave / HW;  // head wave within the token group, token group
  uint16_t* s_tiles = s_kv + tg * NST * TILE;

  const int tok_begin = split * a.split_tokens;
  const int tok_end = min(a.n_tok, tok_begin + a.split_tokens);
  const int rec_begin = tok_begin >> a.tpr_shift;
  const int n_rec = ((tok_end - 1) >> a.tpr_shift) - rec_begin + 1;
  {
    const int32_t* idx_u = a.idx + (int64_t)(unit % a.idx_units) * a.k + rec_begin;
    for (int i = tid; i < n_rec; i += 64 * NW) {
      const int32_t s = idx_u[i];
      s_idx[i] = (s >= 0 && s < a.rec_per_unit) ? s : -1;
    }
  }
  const uint8_t* pool_u = a.pool + (int64_t)unit * a.rec_per_unit * a.R;

  if (tid == 0) s_fallback = 0;
  __syncthreads();  // s_idx is ready
  const int head0 = hb * 32 * HW + hg * 32;  // first head of this wave
  const int head = head0 + col;
  const bool head_ok = head < a.H;
  // Q^T operand: Q[head][16kk + 8 half .. +7], loaded unconditionally (a head past H reads head
  // 0's row: its scores are never stored and, equal to head 0's, change no split-level
  // decision). Unpaced, its loads go out first: they are in flight while the validity masks
  // are written and the first chunks issued. Paced, they follow the first chunks' arrival
  // (below), which spreads the workgroups' start-up traffic.
  bf16x8_t qreg[NKK];
  const uint16_t* qrow = a.q + ((int64_t)unit * a.H + (head_ok ? head : 0)) * DQK + 8 * half;
  auto load_q = [&]() {
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      qreg[kk] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(qrow + kk * 16));
  };
  if constexpr (!PACED) load_q();
  // iteration `it` of token group g covers the split's chunk it * TG + g
  const int n_it = (tok_end - tok_begin + kChunk * TG - 1) / (kChunk * TG);
  // every chunk the groups iterate over gets its word, including a last one wholly past the
  // split end (all zero)
  const int span = n_it * TG * kChunk;
  for (int base = wave * 64; base < span; base += 64 * NW) {
    const int tk = tok_begin + base + lane;
    const bool ok = tk < tok_end && s_idx[(tk >> a.tpr_shift) - rec_begin] >= 0;
    const uint64_t m = __ballot(ok);
    if (lane == 0) {
      s_valid[base >> 5] = (uint32_t)m;
      if (base + 32 < span) s_valid[(base >> 5) + 1] = (uint32_t)(m >> 32);
    }
  }

  const int w_s = __builtin_amdgcn_readfirstlane(hg);
  const int n_loads = w_s < NL_REM ? LPW_MAX : LPW_MIN;
  const int j0 = w_s * LPW_MIN + min(w_s, NL_REM);
  auto chunk_base = [&](int it) { return tok_begin + (it * TG + tg) * kChunk; };
  auto issue = [&](int it, int buf) {
    stage_chunk<P, PP, LPW_MAX>(s_tiles + buf * TILE, s_idx, pool_u, chunk_base(it), tok_end,
                                rec_begin, a.tpr_shift, a.R, a.token_bytes, j0, n_loads);
  };
  f32x16 o[NDV];
#pragma unroll
  for (int n = 0; n < NDV; ++n) o[n] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  float sc[16];

  auto finish_chunk = [&](const uint16_t* tile) {
    uint32_t pw[8];
    float psum = 0.f;
    if (m_run == -INFINITY) {
#pragma unroll
      for (int j = 0; j < 8; ++j) pw[j] = 0u;
    } else {
#pragma unroll
      for (int j = 0; j < 16; j += 2) pw[j >> 1] = weights_bf16x2(sc[j], sc[j + 1], m_run, &psum);
    }
    psum += __shfl_xor(psum, 32, 64);
    l_run += psum;
    const bf16x8_t pa0 = __builtin_bit_cast(bf16x8_t, u32x4{pw[0], pw[1], pw[2], pw[3]});
    const bf16x8_t pa1 = __builtin_bit_cast(bf16x8_t, u32x4{pw[4], pw[5], pw[6], pw[7]});
    // V operand by transpose reads: in each 16-lane group lane 4s+q addresses row
    // 16kb + 4s + half (+2 for the second read), columns 32n + 16 (col >> 4) + 4q .. +3; lane
    // t of the group then holds V[those rows][32n + 16 (col >> 4) + t], the k order of P.
    const uint32_t v0 = lds_addr(tile + (4 * ((lane & 15) >> 2) + half) * PP * 8 +
                                 16 * (col >> 4) + 4 * (lane & 3));
    // MFMA i = (k-step kb, tile n) = (i / NDV, i % NDV), so consecutive MFMAs update
    // different tiles; its two reads run VD MFMAs ahead
    constexpr int VD = 3;
    constexpr int NM = 2 * NDV;
    static_assert(VD == 3 && NM > VD, "the waits below count a ring of 3 read pairs");
    v4i16 vlo[VD], vhi[VD];
    auto vread = [&](int i, int slot) {
      const uint32_t vp = v0 + 2 * ((i / NDV) * 16 * PP * 8 + 32 * (i % NDV));
      vlo[slot] = lds_read_tr16_b64(vp);
      vhi[slot] = lds_read_tr16_b64(vp + 2 * (2 * PP * 8));
    };
#pragma unroll
    for (int i = 0; i < VD; ++i) vread(i, i);
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      // the reads issued after index i's pair: those of indices i+1 .. min(i+VD-1, NM-1)
      const int later = NM - 1 - i < VD - 1 ? NM - 1 - i : VD - 1;
      if (later == 2) lgkm_wait2<4>(vlo[i % VD], vhi[i % VD]);
      else if (later == 1) lgkm_wait2<2>(vlo[i % VD], vhi[i % VD]);
      else lgkm_wait2<0>(vlo[i % VD], vhi[i % VD]);
      const bf16x8_t vb = __builtin_bit_cast(
          bf16x8_t, __builtin_shufflevector(vlo[i % VD], vhi[i % VD], 0, 1, 2, 3, 4, 5, 6, 7));
      o[i % NDV] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(i < NDV ? pa0 : pa1, vb, o[i % NDV],
                                                           0, 0, 0);
      if (i + VD < NM) vread(i + VD, i % VD);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Exponentials are taken against a per-head reference max fixed by the first valid chunk of
  // the split (exact softmax arithmetic with a different reference point; the combine uses the
  // same reference). Scores more than kMlaSlack powers of two above it send the whole split to
  // an exact fallback after the loop, whose results are then discarded; the loop itself never
  // leaves early, so O has a single update path (the MFMAs) and stays in accumulators.
#pragma unroll
  for (int st = 0; st < NST - 1; ++st)
    if (st < n_it) issue(st, st);
  if constexpr (PACED) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    load_q();
  }

  for (int it = 0; it < n_it; ++it) {
    // chunks it+1 .. it+NST-2 were issued earlier and may still be in flight
    wait_chunk<NST, LPW_MAX, LPW_MIN>(min(NST - 2, n_it - 1 - it), w_s < NL_REM);
    const uint16_t* tile = s_tiles + (it % NST) * TILE;
    const int cbase = chunk_base(it);
    // the chunk's validity word, read before the next chunk's loads are issued
    const uint32_t vmask = s_valid[(cbase - tok_begin) >> 5];
    __builtin_amdgcn_sched_barrier(0);
    // every wave is past its reads of buffer (it-1) % NST: refill it with chunk it+NST-1
    if (it + NST - 1 < n_it) issue(it + NST - 1, (it + NST - 1) % NST);

    // ---- scores: S^T for the chunk's 32 tokens x this wave's 32 heads ----
    // K operand reads run KD k-steps ahead of the MFMAs (a small register ring; the
    // scheduling fences keep the compiler from hoisting all 36 reads). The score MFMAs are
    // written as assembly so that their accumulator stays in VGPRs: the output tiles fill
    // the accumulation registers. Hazards hidden from the compiler by the assembly are
    // covered in it: wait states before each MFMA for a just-written operand, and after the
    // last one before the scores are read.
    constexpr int KD = 4;
    static_assert(KD == 4 && NKK > KD, "the waits below count a ring of 4 reads");
    f32x16 sacc, sacc1;  // even / odd k-steps: two independent MFMA chains
    const uint32_t krow = lds_addr(tile + (mla_row(col) * PP + half) * 8);
    u32x4 kbuf[KD];
#pragma unroll
    for (int kk = 0; kk < KD; ++kk) kbuf[kk] = lds_read_b128(krow + kk * 32);
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      // the K reads issued after read kk: those of k-steps kk+1 .. min(kk+KD-1, NKK-1)
      const int later = NKK - 1 - kk < KD - 1 ? NKK - 1 - kk : KD - 1;
      f32x16& acc = (kk & 1) ? sacc1 : sacc;
      if (kk < 2) mfma_qk<KD - 1, true>(acc, kbuf[kk % KD], qreg[kk]);
      else if (later == 3) mfma_qk<3, false>(acc, kbuf[kk % KD], qreg[kk]);
      else if (later == 2) mfma_qk<2, false>(acc, kbuf[kk % KD], qreg[kk]);
      else if (later == 1) mfma_qk<1, false>(acc, kbuf[kk % KD], qreg[kk]);
      else mfma_qk<0, false>(acc, kbuf[kk % KD], qreg[kk]);
      if (kk + KD < NKK) kbuf[kk % KD] = lds_read_b128(krow + (kk + KD) * 32);
      __builtin_amdgcn_sched_barrier(0);
    }
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(sacc), "+v"(sacc1));
    sacc += sacc1;
    int hq = half;
    asm volatile("" : "+v"(hq));
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int bit = mla_row(8 * (j >> 2) + 4 * hq + (j & 3));
      sc[j] = ((vmask >> bit) & 1u) ? sacc[j] * a.scale_log2 : -INFINITY;
    }
    float cmax = sc[0];
#pragma unroll
    for (int j = 1; j < 16; ++j) cmax = fmaxf(cmax, sc[j]);
    cmax = fmaxf(cmax, __shfl_xor(cmax, 32, 64));
    // Validity is per token, so every head of the wave agrees on whether m_run is -inf; while
    // it is, O and l are exactly zero and the reference can simply be set.
    if (m_run == -INFINITY) m_run = cmax;
    else if (__ballot(cmax > m_run + kMlaSlack) && lane == 0) s_fallback = 1;
    finish_chunk(tile);
  }
  wait_loads_and_barrier<0>();  // no staging in flight; s_fallback is final
  if (s_fallback) {
    if (tg == 0)  // the whole split, for this wave's heads
      mla_split_exact(a, s_idx, s_valid, unit, split, tok_begin, tok_end, rec_begin, head0);
    return;
  }
  // ---- partial results of this split, in the accumulator layout (see mla_part_offset) ----
  float* po = a.part_o + ((int64_t)unit * a.n_parts + split) * a.Hp * DV +
              (int64_t)(head0 >> 5) * 32 * DV + lane * 4;
  if constexpr (TG == 2) {
    // The two token groups' results merged per head on the way out, through LDS (the tiles
    // are free now): group 1 leaves its accumulators and (reference max, sum) there; group 0
    // rescales both to the larger reference and adds, in that fixed order, into the stores.
    f32x4* s_o = reinterpret_cast<f32x4*>(s_kv) + hg * 64 * 64;  // [64 regs / 4][64 lanes]
    float2* s_ml = reinterpret_cast<float2*>(reinterpret_cast<f32x4*>(s_kv) + HW * 64 * 64);
    if (tg == 1) {
#pragma unroll
      for (int n = 0; n < NDV; ++n) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          s_o[(n * 4 + q) * 64 + lane] =
              f32x4{o[n][4 * q], o[n][4 * q + 1], o[n][4 * q + 2], o[n][4 * q + 3]};
      }
      if (lane < 32) s_ml[hg * 32 + col] = make_float2(m_run, l_run);
    }
    __syncthreads();
    if (tg == 1) return;
    const float2 other = s_ml[hg * 32 + col];
    const float m_new = fmaxf(m_run, other.x);
    // a group without a valid token has m = -inf, O = 0, l = 0 and contributes nothing
    const float a0 = m_run == -INFINITY ? 0.f : exp2f(m_run - m_new);
    const float a1 = other.x == -INFINITY ? 0.f : exp2f(other.x - m_new);
    l_run = l_run * a0 + other.y * a1;
    m_run = m_new;
    if (head0 < a.H) {
      // Accumulators are read with explicit v_accvgpr_read (arithmetic on them would make the
      // compiler move all of O into VGPRs and spill); the reads are assembly, so the wait states
      // after the last MFMA that wrote them are given here (the barrier above already separates
      // them by far more).
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
      // accumulator row 4q + e of a lane is head 8q + 4 half + e of the wave's 32
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float s0[4], s1[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s0[e] = __shfl(a0, 8 * q + 4 * half + e, 64);
          s1[e] = __shfl(a1, 8 * q + 4 * half + e, 64);
        }
#pragma unroll
        for (int n = 0; n < NDV; ++n) {
          const f32x4 v = s_o[(n * 4 + q) * 64 + lane];
          f32x4 r;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float x;
            asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x) : "a"(o[n][4 * q + e]));
            r[e] = x * s0[e] + v[e] * s1[e];
          }
          *reinterpret_cast<f32x4*>(po + (n * 4 + q) * 256) = r;
        }
      }
    }
  } else if (head0 < a.H) {
#pragma unroll
    for (int n = 0; n < NDV; ++n) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<f32x4*>(po + (n * 4 + q) * 256) =
            f32x4{o[n][4 * q], o[n][4 * q + 1], o[n][4 * q + 2], o[n][4 * q + 3]};
    }
  }
  if (lane < 32 && head_ok)
    a.part_ml[((int64_t)unit * a.n_parts + split) * a.H + head] = make_float2(m_run, l_run);
}

struct CombineArgs {
  const float* part_o;
  const float2* part_ml;
  float* out;
  int32_t H, n_parts, n_rows;  // n_rows = units * H
  int32_t n_wg;                // the merge's own workgroups; those after them run rp
  CarriedReplay rp;
};

// One wave per (unit, head): the largest partial reference max M, the weights
// w_p = 2^(m_p - M), then out = sum_p w_p o_p / sum_p w_p l_p, over the parts in split order.
// Lane j holds the weight of part j of each group of 64 parts; eight parts' outputs are in
// flight at a time.
template <int DV>
__global__ __launch_bounds__(256) void attn_combine_kernel(CombineArgs a) {
  constexpr int E = DV / 64;  // output floats per lane
  static_assert(E == 2 || E == 8, "d_v");
  if ((int)blockIdx.x >= a.n_wg) {  // wave-uniform: the whole workgroup replays
    replay_worker(a.rp, (int)blockIdx.x - a.n_wg);
    return;
  }
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.n_rows) return;
  const int unit = row / a.H, h = row % a.H;
  const int np = a.n_parts;
  const int64_t pstride = (int64_t)a.H * DV;
  const float2* ml = a.part_ml + (int64_t)unit * np * a.H + h;
  const float* po = a.part_o + (int64_t)unit * np * pstride + (int64_t)h * DV + lane * E;

  float M = -INFINITY;
  for (int pb = lane; pb < np; pb += 64) M = fmaxf(M, ml[(int64_t)pb * a.H].x);
#pragma unroll
  for (int x = 32; x >= 1; x >>= 1) M = fmaxf(M, __shfl_xor(M, x, 64));

  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  float lsum = 0.f;
  for (int pb = 0; pb < np; pb += 64) {
    float w = 0.f;
    if (pb + lane < np) {
      const float2 v = ml[(int64_t)(pb + lane) * a.H];
      w = v.x == -INFINITY ? 0.f : exp2f(v.x - M);
      lsum += w * v.y;
    }
    const int n = min(64, np - pb);
    for (int i = 0; i < n; i += 8) {
      float val[8][E];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (i + u < n) {
          const float* src = po + (int64_t)(pb + i + u) * pstride;
#pragma unroll
          for (int e = 0; e < E; e += 2) {
            const float2 t = *reinterpret_cast<const float2*>(src + e);
            val[u][e] = t.x;
            val[u][e + 1] = t.y;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (i + u < n) {
          const float wu = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), i + u));
#pragma unroll
          for (int e = 0; e < E; ++e) acc[e] += wu * val[u][e];
        }
      }
    }
  }
#pragma unroll
  for (int x = 32; x >= 1; x >>= 1) lsum += __shfl_xor(lsum, x, 64);
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  float* dst = a.out + (int64_t)row * DV + lane * E;
#pragma unroll
  for (int e = 0; e < E; e += 2)
    *reinterpret_cast<float2*>(dst + e) = make_float2(acc[e] * inv, acc[e + 1] * inv);
}

struct CombineMlaArgs {
  const float* part_o;    // [units][n_parts][Hp * 512], block layout
  const float2* part_ml;  // [units][n_parts][H]
  float* out;             // [units][H][512]
  int32_t H, Hp, n_parts;
  int32_t n_wg;           // the merge's own workgroups; those after them run rp
  CarriedReplay rp;
};

// Merge of latent-attention partials: one workgroup per (unit, 32-head block, 256 / NS of the
// block's 4096 16-byte groups). Weights w_ph = 2^(m_ph - M_h) and L_h = sum_p w_ph l_ph first
// (in LDS); then thread (slice s, group g) sums parts p = s, s + NS, ... of group g, and the NS
// slice sums are added in slice order (NS > 1 puts more loads in flight when units are few).
template <int NS>
__global__ __launch_bounds__(256) void attn_combine_mla_kernel(CombineMlaArgs a) {
  constexpr int DV = 512, BLK4 = 32 * DV / 4, GPW = 256 / NS;
  __shared__ __align__(16) float s_w[kMlaMaxParts][32];
  __shared__ float s_inv[32];
  __shared__ __align__(16) f32x4 s_acc[NS][GPW];
  if ((int)blockIdx.x >= a.n_wg) {  // wave-uniform: the whole workgroup replays
    replay_worker(a.rp, (int)blockIdx.x - a.n_wg);
    return;
  }
  constexpr int chunks = BLK4 / GPW;
  const int nb = a.Hp >> 5;
  const int chunk = blockIdx.x % chunks;
  const int b = (blockIdx.x / chunks) % nb;
  const int unit = blockIdx.x / (chunks * nb);
  const int t = threadIdx.x, hl = t >> 3, sub = t & 7;
  const int head = b * 32 + hl;
  const int np = a.n_parts;
  const float2* ml = a.part_ml + (int64_t)unit * np * a.H;
  float M = -INFINITY;
  if (head < a.H)
    for (int p = sub; p < np; p += 8) M = fmaxf(M, ml[(int64_t)p * a.H + head].x);
#pragma unroll
  for (int x = 1; x < 8; x <<= 1) M = fmaxf(M, __shfl_xor(M, x, 64));
  float lsum = 0.f;
  for (int p = sub; p < np; p += 8) {
    float w = 0.f;
    if (head < a.H) {
      const float2 v = ml[(int64_t)p * a.H + head];
      w = v.x == -INFINITY ? 0.f : exp2f(v.x - M);
      lsum += w * v.y;
    }
    s_w[p][hl] = w;
  }
#pragma unroll
  for (int x = 1; x < 8; x <<= 1) lsum += __shfl_xor(lsum, x, 64);
  if (sub == 0) s_inv[hl] = lsum > 0.f ? 1.f / lsum : 0.f;
  __syncthreads();

  const int g = t % GPW, sl = t / GPW;
  const int f = chunk * GPW + g;  // 16-byte group within the block
  const int ln = f & 63, q = (f >> 6) & 3, n = f >> 8;
  const int h0 = 8 * q + 4 * (ln >> 5);  // first of the group's four heads (block-local)
  const int64_t pstride = (int64_t)a.Hp * DV;
  const float* pb = a.part_o + (int64_t)unit * np * pstride + (int64_t)b * 32 * DV + 4 * f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  int p = sl;
  for (; p + 3 * NS < np; p += 4 * NS) {
    f32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const f32x4*>(pb + (p + u * NS) * pstride);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      acc += *reinterpret_cast<const f32x4*>(&s_w[p + u * NS][h0]) * v[u];
  }
  for (; p < np; p += NS)
    acc += *reinterpret_cast<const f32x4*>(&s_w[p][h0]) * *reinterpret_cast<const f32x4*>(pb + p * pstride);
  s_acc[sl][g] = acc;
  __syncthreads();
  if (sl == 0) {
    f32x4 r = s_acc[0][g];
#pragma unroll
    for (int s2 = 1; s2 < NS; ++s2) r += s_acc[s2][g];
    const int dim = 32 * n + (ln & 31);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int h = b * 32 + h0 + e;
      if (h < a.H) a.out[((int64_t)unit * a.H + h) * DV + dim] = r[e] * s_inv[h0 + e];
    }
  }
}

// The extra workgroups of a launch that carries a replay: about `threads` threads spread over
// the replay's (unit, layer) pairs, in workgroups of the launch's size `bd`, at most `cap`
// workgroups (at least one per pair). False if the grid would be too large.
bool carried_replay(const FetchArgs& f, int bd, int64_t cap, int32_t threads, int32_t block_bytes,
                    CarriedReplay* r) {
  const int64_t pairs = (int64_t)f.units * f.n_layers;
  int64_t per_pair = std::max<int64_t>(1, threads / (bd * pairs));
  per_pair = std::max<int64_t>(1, std::min(per_pair, cap / pairs));
  if (pairs * per_pair > (1 << 20)) return false;
  r->pf = f;
  r->pf_div = make_fastdiv((uint32_t)(f.R / 16));
  r->pf_per_pair = (int32_t)per_pair;
  r->pf_wg = (int32_t)(pairs * per_pair);
  r->pf_u = std::max(1, block_bytes / 16);
  return true;
}

template <int DQK, int DV, int VOFF, int HW, int TW, int NST>
void launch_partial(const AttnArgs& args, hipStream_t stream) {
  const int nwg_pad = (args.n_wg + 7) & ~7;
  hipLaunchKernelGGL((attn_partial_kernel<DQK, DV, VOFF, HW, TW, NST>), dim3(nwg_pad + args.rp.pf_wg),
                     dim3(64 * HW * TW), 0, stream, args);
}

template <int HW, int TG, int NST, bool PACED = false>
void launch_mla(const AttnArgs& args, hipStream_t stream) {
  const int nwg_pad = (args.n_wg + 7) & ~7;
  hipLaunchKernelGGL((attn_mla_kernel<HW, TG, NST, PACED>), dim3(nwg_pad + args.rp.pf_wg),
                     dim3(64 * HW * TG), 0, stream, args);
}

bool is_mla(const hisparse_attn_desc_t& d) {
  return d.d_qk == 576 && d.d_v == 512 && d.v_offset == 0;
}

}  // namespace

hisparse_status_t plan_attention(int32_t units, int32_t top_k, int32_t record_bytes,
                                 const hisparse_attn_desc_t* attn, AttnPlan* plan) {
  if (!attn || !plan) return HISPARSE_ERR_INVALID_ARG;
  const hisparse_status_t st = hisparse_validate_attn(record_bytes, top_k, attn);
  if (st != HISPARSE_OK) return st;
  if (units <= 0 || (int64_t)units * 256 > (1LL << 30)) return HISPARSE_ERR_INVALID_ARG;
  const int H = attn->q_heads;
  AttnPlan p{};
  p.n_tok = top_k * attn->tokens_per_record;
  if (is_mla(*attn)) {
    // 32 heads per wave; above 32 heads, 2 head waves (64 heads) per workgroup. With 16 or more
    // workgroup columns (units x head blocks) there are enough of them for two token groups per
    // workgroup: twice the tokens per partial result at the same workgroup count, which halves
    // the split partials (fp32, 2 KB per head) and the merge. Measured alone, attention + merge
    // over units of 128 heads (us, best split count): 8 units 27.4 against 28.7, 16 units 34.5
    // against 45.9 (one token group of 4 head waves, 16 splits), 32 units 50.8 against 55.5;
    // below 8 units one token group is faster (2 units 18.7 against 20.7).
    // With HISPARSE_ATTN_BESIDE_FETCH (another stream's host-link fetch shares the GPU) the
    // same shapes take half as many workgroups (below): the other half of the CUs is left to
    // the fetch's waves.
    if (H <= 32) {
      p.hw = 1;
      p.tg = 1;
    } else {
      p.hw = 2;
      p.tg = (int64_t)units * ((H + 63) / 64) >= 16 ? 2 : 1;
    }
    p.tw = 1;
    p.hb = (H + 32 * p.hw - 1) / (32 * p.hw);
  } else {              // up to 64 heads per workgroup, 16 per wave
    p.hw = H > 32 ? 4 : (H > 16 ? 2 : 1);
    p.tw = 4 / p.hw;
    p.tg = 1;
    p.hb = (H + 16 * p.hw - 1) / (16 * p.hw);
  }
  // a split is a whole number of the workgroup's chunk rounds
  const int chunk = kChunk * (is_mla(*attn) ? p.tg : p.tw);
  const int max_splits = (p.n_tok + chunk - 1) / chunk;
  // Beside another stream's host-link fetch, latent attention aims at half a workgroup per CU:
  // the fetch's waves, whose slow host reads occupy the memory pipelines of the CUs they run
  // on, then find CUs without an attention workgroup. Inside the two-micro-batch decode step
  // (16 units of 128 heads, 2 token groups, 4 splits) that fetch moves 51.9 GB/s against 50.6
  // with a workgroup per CU, the step 1.692 against 1.735 ms, and the split partials halve;
  // the attention itself takes 58 against 40 us, hidden behind the other micro-batch's fetch.
  const int target = (is_mla(*attn) && (attn->flags & HISPARSE_ATTN_BESIDE_FETCH))
                         ? kTargetWorkgroups / 2 : kTargetWorkgroups;
  // Beside another stream's fetch and with more than 16 workgroup columns (more than 8 units of
  // 128 heads, two token groups) the call hides behind the other micro-batch's longer fetch,
  // whose host reads then set the step; there every workgroup loading its query together with
  // its first chunks slows those reads, and the paced kernel loads the query after them. The
  // two-micro-batch decode step at 20, 24, 28, 32 and 64 requests took 1.247, 1.450, 1.730,
  // 1.82 and 3.43 ms unpaced against 1.241, 1.371, 1.519, 1.69 and 3.23 ms paced. At 16 columns
  // and below the chain of attention, merge and resolve is the longer one and the unpaced start
  // wins (16 requests: 1.005 against 1.052 ms; 8 requests: 0.711 against 0.724).
  p.paced = is_mla(*attn) && (attn->flags & HISPARSE_ATTN_BESIDE_FETCH) && p.tg == 2 &&
            (int64_t)units * p.hb > 16;
  int splits;
  if (attn->num_splits > 0) {
    splits = std::min(attn->num_splits, max_splits);
  } else {
    // at most one workgroup per CU (a workgroup holds a CU's LDS, so one more would wait for a
    // second round), and enough chunks per split for the load pipeline to reach steady state.
    // For latent attention with one token group the split partials (fp32, 2 KB per head and
    // split) grow with the splits, and longer splits win as the grid gets more workgroup
    // columns: 2 chunks per split up to 4 columns, 4 up to 16, 8 beyond (12 units of 128 heads:
    // 39 against 55 us with 22 two-chunk splits).
    const int per_split = units * p.hb;
    splits = std::max(1, target / per_split);
    int chunks_per_split = 4;
    if (is_mla(*attn)) chunks_per_split = per_split <= 4 ? 2 : (per_split <= 16 ? 4 : 8);
    // A call that carries a replay lasts as long as the replay's host reads; its attention only
    // has to finish within them, and the merge after it is on the decode chain. One request of
    // 128 heads with a replay of its 2048 selections into the next shared layer: 16 four-chunk
    // splits instead of 32 two-chunk ones take the launch from 28.0 to 27.4 us and its merge
    // from 5.8 to 4.6 us (one 1M-token request, 56 layers in groups of 4: decode step 2.299 ->
    // 2.226 ms), although that attention alone takes 17.7 against 12.5 us.
    if (is_mla(*attn) && (attn->flags & HISPARSE_ATTN_CARRIES_REPLAY))
      chunks_per_split = std::max(chunks_per_split, 4);
    // a call too small to give even 64 such workgroups is all latency: one chunk per split
    if (is_mla(*attn) && (int64_t)per_split * (p.n_tok / (2 * chunk)) < 64) chunks_per_split = 1;
    // two token groups: one workgroup per CU, however few chunks each group gets
    if (is_mla(*attn) && p.tg == 2) chunks_per_split = 1;
    const int min_work_splits = std::max(1, p.n_tok / (chunks_per_split * chunk));
    splits = std::max(1, std::min({splits, max_splits, min_work_splits}));
  }
  const int max_split_tokens = std::min(kMaxSplitRecords * attn->tokens_per_record, kMaxSplitTokens);
  splits = std::max(splits, (p.n_tok + max_split_tokens - 1) / max_split_tokens);
  if (is_mla(*attn)) splits = std::min(splits, kMlaMaxParts);  // the merge keeps weights in LDS
  const int per = (p.n_tok + splits - 1) / splits;
  p.split_tokens = (per + chunk - 1) / chunk * chunk;
  if (p.split_tokens > max_split_tokens) p.split_tokens = max_split_tokens / chunk * chunk;
  p.n_wg_splits = (p.n_tok + p.split_tokens - 1) / p.split_tokens;
  p.n_parts = p.n_wg_splits * p.tw;
  // the latent-attention merge holds one weight per part in LDS (hisparse_validate_attn keeps the
  // token count within reach of that limit)
  if (is_mla(*attn) && p.n_parts > kMlaMaxParts) return HISPARSE_ERR_UNSUPPORTED;
  const int64_t n_wg = (int64_t)units * p.n_wg_splits * p.hb;
  if (n_wg > (1LL << 30)) return HISPARSE_ERR_INVALID_ARG;
  const int h_store = is_mla(*attn) ? (H + 31) / 32 * 32 : H;
  const size_t o_bytes = (size_t)units * p.n_parts * h_store * attn->d_v * sizeof(float);
  const size_t ml_bytes = (size_t)units * p.n_parts * H * sizeof(float2);
  p.workspace_bytes = ((o_bytes + 255) & ~(size_t)255) + ml_bytes;
  *plan = p;
  return HISPARSE_OK;
}

hipError_t launch_attention(const AttnPlan& p, const hisparse_attn_desc_t& attn,
                            const uint8_t* pool, int64_t records_per_unit, int32_t record_bytes,
                            int32_t units, int32_t top_k, const uint16_t* q, const int32_t* idx,
                            float* out, void* workspace, hipStream_t stream,
                            int32_t idx_units, const FetchArgs* prefetch,
                            int32_t prefetch_threads, int32_t prefetch_block_bytes) {
  AttnArgs a{};
  if (prefetch && prefetch->units > 0 && prefetch->n_layers > 0) {
    // on the CUs the attention leaves idle (a workgroup of these kernels holds a CU's LDS, so
    // replay and attention never share a CU's memory pipeline)
    const int64_t n_attn = (int64_t)units * p.n_wg_splits * p.hb;
    const int64_t idle = std::max<int64_t>(0, kTargetWorkgroups - ((n_attn + 7) & ~7LL));
    if (!carried_replay(*prefetch, 64 * p.hw * (is_mla(attn) ? p.tg : p.tw), idle,
                        prefetch_threads, prefetch_block_bytes, &a.rp))
      return hipErrorInvalidValue;
  }
  a.idx_units = idx_units > 0 ? idx_units : units;
  a.pool = pool;
  a.q = q;
  a.idx = idx;
  a.Hp = is_mla(attn) ? (attn.q_heads + 31) / 32 * 32 : attn.q_heads;
  const size_t o_bytes = (size_t)units * p.n_parts * a.Hp * attn.d_v * sizeof(float);
  a.part_o = reinterpret_cast<float*>(workspace);
  a.part_ml = reinterpret_cast<float2*>(reinterpret_cast<uint8_t*>(workspace) +
                                        ((o_bytes + 255) & ~(size_t)255));
  a.rec_per_unit = records_per_unit;
  a.R = record_bytes;
  a.token_bytes = record_bytes / attn.tokens_per_record;
  int shift = 0;
  while ((1 << shift) < attn.tokens_per_record) ++shift;
  a.tpr_shift = shift;
  a.k = top_k;
  a.H = attn.q_heads;
  a.n_tok = p.n_tok;
  a.split_tokens = p.split_tokens;
  a.n_wg_splits = p.n_wg_splits;
  a.hb = p.hb;
  a.n_parts = p.n_parts;
  a.n_wg = units * p.n_wg_splits * p.hb;
  a.scale_log2 = attn.scale * 1.4426950408889634f;

  if (is_mla(attn)) {
    if (p.hw == 1) launch_mla<1, 1, 3>(a, stream);
    else if (p.tg == 2 && p.paced) launch_mla<2, 2, 2, true>(a, stream);
    else if (p.tg == 2) launch_mla<2, 2, 2>(a, stream);
    else launch_mla<2, 1, 4>(a, stream);
  } else {
    switch (p.hw) {
      case 1: launch_partial<128, 128, 128, 1, 4, 2>(a, stream); break;
      case 2: launch_partial<128, 128, 128, 2, 2, 3>(a, stream); break;
      default: launch_partial<128, 128, 128, 4, 1, 4>(a, stream); break;
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (attn.flags & HISPARSE_ATTN_DEFER_MERGE) return hipSuccess;
  return launch_merge(p, attn, units, out, workspace, stream);
}

hipError_t launch_merge(const AttnPlan& p, const hisparse_attn_desc_t& attn, int32_t units,
                        float* out, const void* workspace, hipStream_t stream,
                        const FetchArgs* prefetch, int32_t prefetch_threads,
                        int32_t prefetch_block_bytes) {
  // the same workspace layout as launch_attention: partial outputs, then (max, sum) pairs
  const int Hp = is_mla(attn) ? (attn.q_heads + 31) / 32 * 32 : attn.q_heads;
  const size_t o_bytes = (size_t)units * p.n_parts * Hp * attn.d_v * sizeof(float);
  const float* part_o = reinterpret_cast<const float*>(workspace);
  const float2* part_ml = reinterpret_cast<const float2*>(
      reinterpret_cast<const uint8_t*>(workspace) + ((o_bytes + 255) & ~(size_t)255));
  // a carried replay: merge workgroups are small (no CU's whole LDS), so the replay's
  // workgroups run beside them wherever there is room
  CarriedReplay rp{};
  if (prefetch && prefetch->units > 0 && prefetch->n_layers > 0 &&
      !carried_replay(*prefetch, 256, 1 << 20, prefetch_threads, prefetch_block_bytes, &rp))
    return hipErrorInvalidValue;
  if (is_mla(attn)) {
    const int nb = Hp / 32;
    CombineMlaArgs c{part_o, part_ml, out, attn.q_heads, Hp, p.n_parts, 0, rp};
    if ((int64_t)units * nb * 16 >= 2 * kTargetWorkgroups) {
      c.n_wg = units * nb * 16;
      hipLaunchKernelGGL(attn_combine_mla_kernel<1>, dim3(c.n_wg + rp.pf_wg), dim3(256), 0,
                         stream, c);
    } else {
      c.n_wg = units * nb * 64;
      hipLaunchKernelGGL(attn_combine_mla_kernel<4>, dim3(c.n_wg + rp.pf_wg), dim3(256), 0,
                         stream, c);
    }
    return hipGetLastError();
  }
  CombineArgs c{part_o, part_ml, out, attn.q_heads, p.n_parts, units * attn.q_heads, 0, rp};
  c.n_wg = (units * attn.q_heads + 3) / 4;
  hipLaunchKernelGGL(attn_combine_kernel<128>, dim3(c.n_wg + rp.pf_wg), dim3(256), 0, stream, c);
  return hipGetLastError();
}

}  // namespace hisparse
