// Sparse decode attention over gathered records for gfx950 (the consumer of the resolve
// step's slot vector, Section 3.4 Phase 5; exactness per Section 3.1).
//
// For each unit and query head h:  out_h = sum_j softmax_j(scale * q_h . key_j) value_j,
// over the tokens of the k selected records, in the order of the slot vector.
//
// Structure
//   attn_partial_kernel  one workgroup per (unit, token split, head block). A wave owns 16
//     query heads (the MFMA N dimension) and one 32-token chunk per iteration; the workgroup
//     stages its chunk(s) into LDS once and shares them across its head waves.
//       S^T[token][head] = K[token][:] . Q^T[:][head]     v_mfma_f32_16x16x32_bf16, K from LDS
//                                                        rows, Q resident in VGPRs
//       online softmax in fp32 (exp2, running max/sum per head), P rounded to bf16
//       O[head][dim]   += P[head][token] . V[token][dim]  v_mfma_f32_16x16x32_bf16, V^T from
//                                                        LDS (transposed while staging)
//     A lane's S^T accumulator holds tokens {4g..4g+3, 16+4g..16+4g+3} (g = lane/16) of its
//     head, which is exactly one P operand when the PV contraction index runs over the tokens
//     in that order, so P never leaves the lane; the V^T operand is read in the same order.
//   attn_combine_kernel  merges the per-split (max, sum, unnormalised output) triples of each
//     (unit, head) in ascending split order.
// The reduction order depends only on token positions in the sequence, never on the slot
// values, so any placement of the same records gives bit-identical outputs.
#include <math.h>

#include "internal.h"

namespace hisparse {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kChunk = 32;            // tokens per wave per iteration
constexpr int kKPad = 8;              // bf16 padding per K row in LDS
constexpr int kVtRow = kChunk + 8;    // bf16 per V^T row in LDS (32 tokens + padding)
constexpr int kTargetWorkgroups = 512;

struct AttnArgs {
  const uint8_t* pool;
  const uint16_t* q;
  const int32_t* idx;
  float* part_o;    // [units][n_parts][H][DV]
  float2* part_ml;  // [units][n_parts][H] (running max in log2 units, running sum)
  int64_t rec_per_unit;
  int32_t R, token_bytes, tpr_shift, k, H, n_tok;
  int32_t split_tokens, n_wg_splits, hb, n_parts, n_wg;
  float scale_log2;
};

__device__ inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ inline u32x4 lds_load16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ inline u32x2 lds_load8(const uint16_t* p) { return *reinterpret_cast<const u32x2*>(p); }
__device__ inline void lds_store16(uint16_t* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// Key chunks (8 bf16 each) that the value range does not already cover.
template <int DQK, int DV, int VOFF>
struct KeyOnly {
  static_assert(VOFF == 0 || VOFF >= DQK, "value range must start the token or follow the key");
  static constexpr int start = VOFF == 0 ? DV / 8 : 0;
  static constexpr int count = VOFF == 0 ? DQK / 8 - DV / 8 : DQK / 8;
};

template <int DQK, int DV, int VOFF, int HW, int TW>
__global__ __launch_bounds__(64 * HW * TW) void attn_partial_kernel(AttnArgs a) {
  constexpr int GT = 64 * HW;                 // threads per token group
  constexpr int KROW = DQK + kKPad;
  constexpr int K_TILE = kChunk * KROW;
  constexpr int VT_TILE = DV * kVtRow;
  constexpr int TG_ELEMS = K_TILE + VT_TILE;
  constexpr int NKK = DQK / 32;
  constexpr int NOUT = DV / 16;
  constexpr int VCH = DV / 8;                 // value chunks per token
  using KO = KeyOnly<DQK, DV, VOFF>;
  static_assert(DQK % 32 == 0 && DV % 16 == 0, "shape");
  __shared__ __align__(16) uint16_t s_kv[TW * TG_ELEMS];

  // XCD-aware mapping: consecutive workgroup ids go round-robin over the 8 XCDs, so give each
  // XCD a contiguous range of work items; the head blocks of one (unit, split) then share the
  // staged records through the same L2.
  const int nwg_pad = (a.n_wg + 7) & ~7;
  const int w = (int)(blockIdx.x & 7) * (nwg_pad >> 3) + (int)(blockIdx.x >> 3);
  if (w >= a.n_wg) return;
  const int hb = w % a.hb;
  const int split = (w / a.hb) % a.n_wg_splits;
  const int unit = w / (a.hb * a.n_wg_splits);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hg = wave % HW, tg = wave / HW;
  const int gtid = tid - tg * GT;
  const int g = lane >> 4;
  uint16_t* s_k = s_kv + tg * TG_ELEMS;
  uint16_t* s_vt = s_k + K_TILE;

  const int head = hb * 16 * HW + hg * 16 + (lane & 15);
  const bool head_ok = head < a.H;
  bf16x8_t qreg[NKK];
  {
    const uint16_t* qrow = a.q + ((int64_t)unit * a.H + (head_ok ? head : 0)) * DQK + 8 * g;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (head_ok) v = *reinterpret_cast<const u32x4*>(qrow + kk * 32);
      qreg[kk] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  f32x4 o[NOUT];
#pragma unroll
  for (int n = 0; n < NOUT; ++n) o[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const int tok_begin = split * a.split_tokens;
  const int tok_end = min(a.n_tok, tok_begin + a.split_tokens);
  const int32_t* idx_u = a.idx + (int64_t)unit * a.k;
  const uint8_t* pool_u = a.pool + (int64_t)unit * a.rec_per_unit * a.R;
  const int tpr_mask = (1 << a.tpr_shift) - 1;

  for (int c0 = tok_begin; c0 < tok_end; c0 += kChunk * TW) {
    const int cbase = c0 + tg * kChunk;
    __syncthreads();  // the previous chunk's LDS reads are done

    // ---- stage: K rows natural, V transposed to [dim][token] ----
    for (int item = gtid; item < (kChunk / 8) * VCH; item += GT) {
      const int oct = item / VCH, c = item % VCH;
      u32x4 in[8];
#pragma unroll
      for (int t8 = 0; t8 < 8; ++t8) {
        const int tk = cbase + oct * 8 + t8;
        in[t8] = u32x4{0u, 0u, 0u, 0u};
        if (tk < tok_end) {
          const int32_t s = idx_u[tk >> a.tpr_shift];
          if (s >= 0 && s < a.rec_per_unit)
            in[t8] = *reinterpret_cast<const u32x4*>(pool_u + (int64_t)s * a.R +
                                                     (int64_t)(tk & tpr_mask) * a.token_bytes +
                                                     (VOFF + c * 8) * 2);
        }
      }
      if (VOFF + c * 8 < DQK) {
#pragma unroll
        for (int t8 = 0; t8 < 8; ++t8) lds_store16(s_k + (oct * 8 + t8) * KROW + VOFF + c * 8, in[t8]);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        u32x4 r;
#pragma unroll
        for (int w2 = 0; w2 < 4; ++w2) {
          const uint32_t x = in[2 * w2][j >> 1], y = in[2 * w2 + 1][j >> 1];
          r[w2] = (j & 1) ? ((x >> 16) | (y & 0xFFFF0000u)) : ((x & 0xFFFFu) | (y << 16));
        }
        lds_store16(s_vt + (c * 8 + j) * kVtRow + oct * 8, r);
      }
    }
    for (int item = gtid; item < kChunk * KO::count; item += GT) {
      const int tok = item / KO::count, c = KO::start + item % KO::count;
      const int tk = cbase + tok;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (tk < tok_end) {
        const int32_t s = idx_u[tk >> a.tpr_shift];
        if (s >= 0 && s < a.rec_per_unit)
          v = *reinterpret_cast<const u32x4*>(pool_u + (int64_t)s * a.R +
                                              (int64_t)(tk & tpr_mask) * a.token_bytes + c * 16);
      }
      lds_store16(s_k + tok * KROW + c * 8, v);
    }
    __syncthreads();

    // ---- scores: S^T tiles for tokens [0,16) and [16,32) of the chunk ----
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
    const uint16_t* k0 = s_k + (lane & 15) * KROW + 8 * g;
    const uint16_t* k1 = k0 + 16 * KROW;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const bf16x8_t a0 = __builtin_bit_cast(bf16x8_t, lds_load16(k0 + kk * 32));
      const bf16x8_t a1 = __builtin_bit_cast(bf16x8_t, lds_load16(k1 + kk * 32));
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, qreg[kk], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, qreg[kk], s1, 0, 0, 0);
    }

    // ---- online softmax for this lane's head over its 8 tokens ----
    float sc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int tk = cbase + (j < 4 ? 4 * g + j : 16 + 4 * g + (j - 4));
      bool ok = tk < tok_end;
      if (ok) {
        const int32_t s = idx_u[tk >> a.tpr_shift];
        ok = s >= 0 && s < a.rec_per_unit;
      }
      const float raw = j < 4 ? s0[j] : s1[j - 4];
      sc[j] = ok ? raw * a.scale_log2 : -INFINITY;
    }
    float cmax = sc[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) cmax = fmaxf(cmax, sc[j]);
    cmax = fmaxf(cmax, __shfl_xor(cmax, 16, 64));
    cmax = fmaxf(cmax, __shfl_xor(cmax, 32, 64));
    const float m_new = fmaxf(m_run, cmax);
    float alpha = 1.f;
    uint32_t pw[4];
    float psum = 0.f;
    if (m_new == -INFINITY) {
      pw[0] = pw[1] = pw[2] = pw[3] = 0u;
    } else {
      alpha = exp2f(m_run - m_new);
#pragma unroll
      for (int j = 0; j < 8; j += 2) {
        const uint16_t b0 = f32_to_bf16_rne(exp2f(sc[j] - m_new));
        const uint16_t b1 = f32_to_bf16_rne(exp2f(sc[j + 1] - m_new));
        psum += bf16_to_f32(b0);
        psum += bf16_to_f32(b1);
        pw[j >> 1] = (uint32_t)b0 | ((uint32_t)b1 << 16);
      }
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;

    // ---- rescale O rows (heads 4g..4g+3) and accumulate P . V ----
    float al[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) al[j] = __shfl(alpha, 4 * g + j, 64);
#pragma unroll
    for (int n = 0; n < NOUT; ++n) {
#pragma unroll
      for (int j = 0; j < 4; ++j) o[n][j] *= al[j];
    }
    const bf16x8_t pa = __builtin_bit_cast(bf16x8_t, u32x4{pw[0], pw[1], pw[2], pw[3]});
    const uint16_t* vt = s_vt + (lane & 15) * kVtRow + 4 * g;
#pragma unroll
    for (int n = 0; n < NOUT; ++n) {
      const uint16_t* r = vt + n * 16 * kVtRow;
      const u32x2 lo = lds_load8(r), hi = lds_load8(r + 16);
      const bf16x8_t vb = __builtin_bit_cast(bf16x8_t, u32x4{lo[0], lo[1], hi[0], hi[1]});
      o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vb, o[n], 0, 0, 0);
    }
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

struct CombineArgs {
  const float* part_o;
  const float2* part_ml;
  float* out;
  int32_t H, n_parts;
};

template <int DV>
__global__ __launch_bounds__(DV / 4) void attn_combine_kernel(CombineArgs a) {
  const int uh = blockIdx.x;
  const int unit = uh / a.H, h = uh % a.H;
  const float2* ml = a.part_ml + (int64_t)unit * a.n_parts * a.H + h;
  float M = -INFINITY;
  for (int p = 0; p < a.n_parts; ++p) M = fmaxf(M, ml[(int64_t)p * a.H].x);
  float lsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  const int d = threadIdx.x * 4;
  for (int p = 0; p < a.n_parts; ++p) {
    const float2 v = ml[(int64_t)p * a.H];
    const float wgt = v.x == -INFINITY ? 0.f : exp2f(v.x - M);
    lsum += wgt * v.y;
    const f32x4 po = *reinterpret_cast<const f32x4*>(
        a.part_o + (((int64_t)unit * a.n_parts + p) * a.H + h) * DV + d);
    acc += wgt * po;
  }
  f32x4 r = {0.f, 0.f, 0.f, 0.f};
  if (lsum > 0.f) r = acc / lsum;
  *reinterpret_cast<f32x4*>(a.out + ((int64_t)unit * a.H + h) * DV + d) = r;
}

template <int DQK, int DV, int VOFF, int HW, int TW>
void launch_partial(const AttnArgs& args, hipStream_t stream) {
  const int nwg_pad = (args.n_wg + 7) & ~7;
  hipLaunchKernelGGL((attn_partial_kernel<DQK, DV, VOFF, HW, TW>), dim3(nwg_pad),
                     dim3(64 * HW * TW), 0, stream, args);
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
  p.hw = H <= 16 ? 1 : (H <= 32 ? 2 : 4);
  p.tw = is_mla(*attn) ? 1 : 4 / p.hw;
  p.hb = (H + 16 * p.hw - 1) / (16 * p.hw);
  p.n_tok = top_k * attn->tokens_per_record;
  const int chunk = kChunk * p.tw;
  const int max_splits = (p.n_tok + chunk - 1) / chunk;
  int splits;
  if (attn->num_splits > 0) {
    splits = std::min(attn->num_splits, max_splits);
  } else {
    const int per_split = units * p.hb;
    splits = (kTargetWorkgroups + per_split - 1) / per_split;
    splits = std::max(1, std::min(splits, max_splits));
  }
  const int per = (p.n_tok + splits - 1) / splits;
  p.split_tokens = (per + chunk - 1) / chunk * chunk;
  p.n_wg_splits = (p.n_tok + p.split_tokens - 1) / p.split_tokens;
  p.n_parts = p.n_wg_splits * p.tw;
  const int64_t n_wg = (int64_t)units * p.n_wg_splits * p.hb;
  if (n_wg > (1LL << 30)) return HISPARSE_ERR_INVALID_ARG;
  const size_t o_bytes = (size_t)units * p.n_parts * H * attn->d_v * sizeof(float);
  const size_t ml_bytes = (size_t)units * p.n_parts * H * sizeof(float2);
  p.workspace_bytes = ((o_bytes + 255) & ~(size_t)255) + ml_bytes;
  *plan = p;
  return HISPARSE_OK;
}

hipError_t launch_attention(const AttnPlan& p, const hisparse_attn_desc_t& attn,
                            const uint8_t* pool, int64_t records_per_unit, int32_t record_bytes,
                            int32_t units, int32_t top_k, const uint16_t* q, const int32_t* idx,
                            float* out, void* workspace, hipStream_t stream) {
  AttnArgs a{};
  a.pool = pool;
  a.q = q;
  a.idx = idx;
  const size_t o_bytes = (size_t)units * p.n_parts * attn.q_heads * attn.d_v * sizeof(float);
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
    switch (p.hw) {
      case 1: launch_partial<576, 512, 0, 1, 1>(a, stream); break;
      case 2: launch_partial<576, 512, 0, 2, 1>(a, stream); break;
      default: launch_partial<576, 512, 0, 4, 1>(a, stream); break;
    }
  } else {
    switch (p.hw) {
      case 1: launch_partial<128, 128, 128, 1, 4>(a, stream); break;
      case 2: launch_partial<128, 128, 128, 2, 2>(a, stream); break;
      default: launch_partial<128, 128, 128, 4, 1>(a, stream); break;
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  CombineArgs c{a.part_o, a.part_ml, out, attn.q_heads, p.n_parts};
  if (attn.d_v == 512)
    hipLaunchKernelGGL(attn_combine_kernel<512>, dim3(units * attn.q_heads), dim3(128), 0, stream, c);
  else
    hipLaunchKernelGGL(attn_combine_kernel<128>, dim3(units * attn.q_heads), dim3(32), 0, stream, c);
  return hipGetLastError();
}

}  // namespace hisparse
