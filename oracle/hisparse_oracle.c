/*
 * HiSparse CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded reference for what the HiSparse decode hot path computes.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may load it; the
 * product library never does. It shares no code with the HIP library.
 *
 * What it implements (paper: "HiSparse: Scaling Sparse-Attention Decoding with Hierarchical
 * KV Cache Management"):
 *
 *  - oracle_resolve: one step of miss resolution for one cache unit (one request-layer cache,
 *    or one request-layer-kv-head cache). The data model is Section 3.2 ("KV Hierarchy and
 *    Metadata"): B slots, a page table mapping each logical record to a slot or to a host-only
 *    sentinel, and LRU recency metadata. The replacement rule is Section 3.2 "Replacement
 *    policy" with Section 3.4 Phase 3: plain LRU among slots the current step does not
 *    reference, with the step's hits promoted above the step's newly fetched misses. The
 *    paper fixes no tie-break; the oracle uses the canonical deterministic reading:
 *      * timestamps: misses of step t get 2t-1 and hits get 2t, so both outrank every earlier
 *        step and hits outrank same-step misses;
 *      * victims are the non-hit slots in ascending (timestamp, slot) order; empty slots have
 *        timestamp 0 and so are consumed first, in slot order;
 *      * the i-th miss in ascending position order takes the i-th victim.
 *    Output (Section 3.3 (3), Section 3.4 Phase 5): for each input index i, the slot now
 *    holding sel[i] ("top-k order"), plus (hits, misses) and the miss plan (position -> slot)
 *    that Section 3.5 replays into shared layers.
 *  - oracle_apply_plan: Section 3.4 Phase 4, the copy of each missed host record into its slot.
 *  - oracle_sparse_decode: Section 3.1 "Exact sparse-attention outputs": softmax attention of
 *    each query head over the tokens of the selected records, in float64, read from whatever
 *    pool the indices address (the full host KV, or the GPU-cache image through slots).
 *
 * Readings where the paper is silent: negative selection entries are padding (output slot -1,
 * not counted); an entry outside [0, L) or a repeated entry makes the whole selection invalid,
 * in which case the unit's state is left unchanged, every output slot is -1, counts are
 * (0, 0) and ORACLE_BAD_SELECTION is returned. The step clock advances only on valid calls.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_BAD_SELECTION (-5)
#define ORACLE_INVALID_ARG (-1)
#define ORACLE_OOM (-2)

static int cmp_i32(const void* a, const void* b) {
  int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  return (x > y) - (x < y);
}

typedef struct { uint32_t ts; int32_t slot; } cand_t;

static int cmp_cand(const void* a, const void* b) {
  const cand_t* x = (const cand_t*)a;
  const cand_t* y = (const cand_t*)b;
  if (x->ts != y->ts) return (x->ts > y->ts) - (x->ts < y->ts);
  return (x->slot > y->slot) - (x->slot < y->slot);
}

/* One resolve step for one unit. State arrays: pt[L] (slot or -1), slot_pos[B] (position or -1),
 * slot_ts[B], *clock (valid steps so far). Outputs: slots_out[k], counts_out[2] = {hits, misses},
 * plan_pos/plan_slot[misses] (may be NULL). */
int oracle_resolve(int64_t L, int32_t B, int32_t k, int32_t* pt, int32_t* slot_pos,
                   uint32_t* slot_ts, uint32_t* clock, const int32_t* sel, int32_t* slots_out,
                   int32_t* counts_out, int32_t* plan_pos, int32_t* plan_slot) {
  if (L <= 0 || B <= 0 || k < 0 || k > B) return ORACLE_INVALID_ARG;
  int32_t* valid = malloc(sizeof(int32_t) * (size_t)(k + 1));
  int32_t* misses = malloc(sizeof(int32_t) * (size_t)(k + 1));
  unsigned char* hit_slot = calloc((size_t)B, 1);
  cand_t* cand = malloc(sizeof(cand_t) * (size_t)B);
  int rc = ORACLE_OK;
  if (!valid || !misses || !hit_slot || !cand) { rc = ORACLE_OOM; goto done; }

  /* the selected set S: non-negative entries, which must lie in [0, L) and be distinct */
  int32_t n_valid = 0;
  for (int32_t i = 0; i < k; ++i) {
    if (sel[i] < 0) continue;
    if ((int64_t)sel[i] >= L) { rc = ORACLE_BAD_SELECTION; break; }
    valid[n_valid++] = sel[i];
  }
  if (rc == ORACLE_OK) {
    qsort(valid, (size_t)n_valid, sizeof(int32_t), cmp_i32);
    for (int32_t i = 1; i < n_valid; ++i)
      if (valid[i] == valid[i - 1]) { rc = ORACLE_BAD_SELECTION; break; }
  }
  if (rc != ORACLE_OK) {
    for (int32_t i = 0; i < k; ++i) slots_out[i] = -1;
    counts_out[0] = counts_out[1] = 0;
    goto done;
  }

  const uint32_t t = *clock + 1;
  /* hits: selected positions already resident; misses: the rest, ascending (valid is sorted) */
  int32_t n_hit = 0, n_miss = 0;
  for (int32_t i = 0; i < n_valid; ++i) {
    int32_t s = pt[valid[i]];
    if (s >= 0) { hit_slot[s] = 1; ++n_hit; }
    else misses[n_miss++] = valid[i];
  }
  /* hits are promoted to the most-recent end */
  for (int32_t s = 0; s < B; ++s)
    if (hit_slot[s]) slot_ts[s] = 2u * t;
  /* victims: slots not hit this step, least recent first, ties by slot index */
  int32_t n_cand = 0;
  for (int32_t s = 0; s < B; ++s)
    if (!hit_slot[s]) cand[n_cand++] = (cand_t){slot_ts[s], s};
  qsort(cand, (size_t)n_cand, sizeof(cand_t), cmp_cand);
  if (n_miss > n_cand) { rc = ORACLE_INVALID_ARG; goto done; } /* impossible when k <= B */
  for (int32_t i = 0; i < n_miss; ++i) {
    int32_t v = cand[i].slot, p = misses[i];
    if (slot_pos[v] >= 0) pt[slot_pos[v]] = -1; /* evicted record becomes host-only */
    slot_pos[v] = p;
    pt[p] = v;
    slot_ts[v] = 2u * t - 1u; /* fetched misses sit just behind this step's hits */
    if (plan_pos) plan_pos[i] = p;
    if (plan_slot) plan_slot[i] = v;
  }
  for (int32_t i = 0; i < k; ++i) slots_out[i] = sel[i] >= 0 ? pt[sel[i]] : -1;
  counts_out[0] = n_hit;
  counts_out[1] = n_miss;
  *clock = t;
done:
  free(valid); free(misses); free(hit_slot); free(cand);
  return rc;
}

/* oracle_resolve over n_units units laid out contiguously: pt[u*L], slot_pos/slot_ts[u*B],
 * clock[u], sel/slots_out/plan_*[u*k], counts_out[u*2]. Returns the number of units whose
 * selection was invalid, or a negative argument error. */
int oracle_resolve_units(int32_t n_units, int64_t L, int32_t B, int32_t k, int32_t* pt,
                         int32_t* slot_pos, uint32_t* slot_ts, uint32_t* clock,
                         const int32_t* sel, int32_t* slots_out, int32_t* counts_out,
                         int32_t* plan_pos, int32_t* plan_slot) {
  int bad = 0;
  for (int32_t u = 0; u < n_units; ++u) {
    int rc = oracle_resolve(L, B, k, pt + (int64_t)u * L, slot_pos + (int64_t)u * B,
                            slot_ts + (int64_t)u * B, clock + u, sel + (int64_t)u * k,
                            slots_out + (int64_t)u * k, counts_out + 2 * (int64_t)u,
                            plan_pos ? plan_pos + (int64_t)u * k : NULL,
                            plan_slot ? plan_slot + (int64_t)u * k : NULL);
    if (rc == ORACLE_BAD_SELECTION) ++bad;
    else if (rc != ORACLE_OK) return rc;
  }
  return bad;
}

/* Phase 4: cache[plan_slot[i]] <- host[plan_pos[i]], R bytes each. */
void oracle_apply_plan(const uint8_t* host, uint8_t* cache, int32_t R, const int32_t* plan_pos,
                       const int32_t* plan_slot, int32_t m) {
  for (int32_t i = 0; i < m; ++i)
    memcpy(cache + (int64_t)plan_slot[i] * R, host + (int64_t)plan_pos[i] * R, (size_t)R);
}

static double bf16_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* Sparse decode attention for one unit, float64.
 * q[H][d_qk] bf16; pool[*][tokens_per_record * token_elems] bf16, record r at
 * pool + r * tokens_per_record * token_elems; idx[k] record indices (-1 = padding).
 * Token j of the attended sequence is token (j % tpr) of record idx[j / tpr]; key = its first
 * d_qk elements, value = d_v elements from v_off. out[H][d_v]:
 *   out_h = sum_j softmax_j(scale * <q_h, key_j>) value_j, tokens in selection order.
 * With no valid token the output is zero. */
int oracle_sparse_decode(const uint16_t* q, int32_t H, int32_t d_qk, int32_t d_v, int32_t v_off,
                         int32_t token_elems, int32_t tokens_per_record, const uint16_t* pool,
                         const int32_t* idx, int32_t k, double scale, double* out) {
  if (H <= 0 || d_qk <= 0 || d_v <= 0 || v_off < 0 || d_qk > token_elems ||
      v_off + d_v > token_elems || tokens_per_record <= 0 || k < 0)
    return ORACLE_INVALID_ARG;
  const int64_t rec_elems = (int64_t)tokens_per_record * token_elems;
  int64_t n_tok = 0;
  for (int32_t i = 0; i < k; ++i) n_tok += idx[i] >= 0 ? tokens_per_record : 0;
  const uint16_t** tok = malloc(sizeof(uint16_t*) * (size_t)(n_tok + 1));
  double* s = malloc(sizeof(double) * (size_t)(n_tok + 1));
  double* qd = malloc(sizeof(double) * (size_t)d_qk);
  if (!tok || !s || !qd) { free(tok); free(s); free(qd); return ORACLE_OOM; }
  int64_t n = 0;
  for (int32_t i = 0; i < k; ++i) {
    if (idx[i] < 0) continue;
    for (int32_t t = 0; t < tokens_per_record; ++t)
      tok[n++] = pool + (int64_t)idx[i] * rec_elems + (int64_t)t * token_elems;
  }
  for (int32_t h = 0; h < H; ++h) {
    double* o = out + (int64_t)h * d_v;
    for (int32_t d = 0; d < d_v; ++d) o[d] = 0.0;
    if (n_tok == 0) continue;
    for (int32_t d = 0; d < d_qk; ++d) qd[d] = bf16_to_double(q[(int64_t)h * d_qk + d]);
    double mx = -INFINITY;
    for (int64_t j = 0; j < n_tok; ++j) {
      double acc = 0.0;
      for (int32_t d = 0; d < d_qk; ++d) acc += qd[d] * bf16_to_double(tok[j][d]);
      s[j] = scale * acc;
      if (s[j] > mx) mx = s[j];
    }
    double z = 0.0;
    for (int64_t j = 0; j < n_tok; ++j) { s[j] = exp(s[j] - mx); z += s[j]; }
    for (int64_t j = 0; j < n_tok; ++j) {
      const double w = s[j] / z;
      const uint16_t* v = tok[j] + v_off;
      for (int32_t d = 0; d < d_v; ++d) o[d] += w * bf16_to_double(v[d]);
    }
  }
  free(tok); free(s); free(qd);
  return ORACLE_OK;
}
