/*
 * oracle.c -- plain, slow CPU oracle of the M2Cache decode hot path
 * (arXiv 2410.14740): predictor scores, top-k with score-rank precision tiers,
 * the per-layer neuron slot cache with LRU replacement, and the sparse
 * mixed-precision SwiGLU FFN.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link or call it;
 * only the tests, the smoke check and the benchmark's CPU-baseline leg do.
 * It shares no code with the HIP library: every step below is written out
 * from its definition, in loops, in the order the definition gives.
 *
 * Build: gcc -O2 -std=c99 -ffp-contract=off -fopenmp -fPIC -shared oracle.c -lm
 * (no fast-math and no FMA contraction: every fused multiply-add below is an
 * explicit fmaf call). OpenMP only splits independent results over threads:
 * every dot product and every output element is still one sum taken in the
 * order its definition gives, so the results do not depend on the thread
 * count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Threads the oracle may use (1 = the serial program). */
void orc_set_threads(int n) {
#ifdef _OPENMP
  omp_set_num_threads(n > 0 ? n : 1);
#else
  (void)n;
#endif
}

int orc_get_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* IEEE binary16 <-> binary32, written from the format definition.           */
/* Weights, predictor and activations are fp16; scales are fp16 (the
 * quantization scheme the workload fixes: symmetric, group 128, fp16 scales).*/

float orc_f16_to_f32(uint16_t h) {
  int sign = (h >> 15) & 1;
  int exp = (h >> 10) & 0x1f;
  int man = h & 0x3ff;
  double v;
  if (exp == 0) {
    v = ldexp((double)man, -24); /* subnormal: man * 2^-24 */
  } else if (exp == 31) {
    v = man ? NAN : INFINITY;
  } else {
    v = ldexp((double)(1024 + man), exp - 25); /* (1 + man/1024) * 2^(exp-15) */
  }
  return (float)(sign ? -v : v); /* exact: at most 11 significant bits */
}

/* Round-to-nearest-even conversion. */
uint16_t orc_f32_to_f16(float f) {
  uint16_t sign = signbit(f) ? 0x8000 : 0;
  double a = fabs((double)f);
  if (isnan(f)) return sign | 0x7e00;
  if (a >= 65520.0) return sign | 0x7c00; /* 65520 is the tie between 65504 and 2^16 */
  if (a < ldexp(1.0, -14)) {
    /* subnormal range: quantum 2^-24; m == 1024 is the smallest normal. */
    double m = nearbyint(a * ldexp(1.0, 24)); /* exact scaling, RNE */
    return sign | (uint16_t)m;
  }
  int e2;
  frexp(a, &e2);                 /* a = f * 2^e2, f in [0.5, 1): exponent e2-1 */
  int e = e2 - 1;                /* -14 <= e <= 15 */
  double m = nearbyint(ldexp(a, 10 - e)); /* in [1024, 2048] */
  if (m == 2048.0) { m = 1024.0; e += 1; }
  if (e > 15) return sign | 0x7c00;
  return sign | (uint16_t)(((e + 15) << 10) | ((int)m - 1024));
}

/* ------------------------------------------------------------------------ */
/* Neuron records (Sec. 1 footnote and Sec. 5.2: a neuron is row i of the
 * gate and up matrices plus column i of the down matrix; lower-scored
 * neurons are loaded at lower precision). Layout of one record:
 *   FP16: gate[d] up[d] down[d] as fp16                      (6d bytes)
 *   INT8: gate[d] up[d] down[d] int8, then G fp16 scales per vector
 *   INT4: gate[d/2] up[d/2] down[d/2] packed two's-complement nibbles
 *         (element 2m low nibble of byte m), then G scales per vector
 * G = d/128.                                                              */

int64_t orc_record_bytes(int d, int tier) {
  int64_t G = d / 128;
  if (tier == 3) return 6LL * d;
  if (tier == 2) return 3LL * d + 6 * G;
  if (tier == 1) return 3LL * d / 2 + 6 * G;
  return -1;
}

/* Quantize one group of n fp16 weights symmetrically with qmax levels each
 * side: s = fp16(fp32(amax) / qmax), q = clamp(rne(w / s)), q = 0 if s == 0. */
static void quant_group(const float* w, int n, int qmax, int* q, uint16_t* s_bits) {
  float amax = 0.0f;
  for (int j = 0; j < n; j++) {
    float a = fabsf(w[j]);
    if (a > amax) amax = a;
  }
  float sq = amax / (float)qmax; /* IEEE fp32 division */
  uint16_t sb = orc_f32_to_f16(sq);
  float s = orc_f16_to_f32(sb);
  for (int j = 0; j < n; j++) {
    int v = 0;
    if (s != 0.0f) {
      float r = rintf(w[j] / s); /* fp32 quotient, round half to even */
      if (r > (float)qmax) r = (float)qmax;
      if (r < -(float)qmax) r = -(float)qmax;
      v = (int)r;
    }
    q[j] = v;
  }
  *s_bits = sb;
}

/* Build the tier-`tier` record of every neuron. w_gate, w_up [d_ff][d];
 * w_down [d][d_ff]; out [d_ff][stride]. Returns 0, or -1 on bad arguments. */
int orc_build_records(int d, int d_ff, const uint16_t* w_gate, const uint16_t* w_up,
                      const uint16_t* w_down, int tier, uint8_t* out, int64_t stride) {
  if (d <= 0 || d % 128 != 0 || d_ff <= 0 || tier < 1 || tier > 3) return -1;
  if (stride < orc_record_bytes(d, tier)) return -1;
  int G = d / 128;
#pragma omp parallel
  {
  float* vec = (float*)malloc(sizeof(float) * d);
  int* q = (int*)malloc(sizeof(int) * d);
#pragma omp for schedule(dynamic, 16)
  for (int i = 0; i < d_ff; i++) {
    uint8_t* rec = out + (int64_t)i * stride;
    memset(rec, 0, (size_t)stride);
    for (int v = 0; v < 3; v++) { /* 0 gate, 1 up, 2 down */
      /* gather the vector as fp16 bits */
      for (int j = 0; j < d; j++) {
        uint16_t hb;
        if (v == 0) hb = w_gate[(int64_t)i * d + j];
        else if (v == 1) hb = w_up[(int64_t)i * d + j];
        else hb = w_down[(int64_t)j * d_ff + i];
        if (tier == 3) {
          rec[(int64_t)v * 2 * d + 2 * j] = (uint8_t)(hb & 0xff);
          rec[(int64_t)v * 2 * d + 2 * j + 1] = (uint8_t)(hb >> 8);
        }
        vec[j] = orc_f16_to_f32(hb);
      }
      if (tier == 3) continue;
      int qmax = (tier == 2) ? 127 : 7;
      int64_t codes_bytes = (tier == 2) ? d : d / 2; /* per vector */
      uint8_t* codes = rec + v * codes_bytes;
      uint8_t* scales = rec + 3 * codes_bytes + (int64_t)v * 2 * G;
      for (int g = 0; g < G; g++) {
        uint16_t sb;
        quant_group(vec + g * 128, 128, qmax, q + g * 128, &sb);
        scales[2 * g] = (uint8_t)(sb & 0xff);
        scales[2 * g + 1] = (uint8_t)(sb >> 8);
      }
      for (int j = 0; j < d; j++) {
        if (tier == 2) {
          codes[j] = (uint8_t)(int8_t)q[j];
        } else {
          uint8_t nib = (uint8_t)(q[j] & 0xf);
          if (j % 2 == 0) codes[j / 2] |= nib;
          else codes[j / 2] |= (uint8_t)(nib << 4);
        }
      }
    }
  }
  free(vec);
  free(q);
  }
  return 0;
}

/* Exact dequantized values of elements [j0, j0 + n) of vector v (0 gate,
 * 1 up, 2 down) of one record. */
static void dequant_part(int d, int tier, const uint8_t* rec, int v, int j0, int n, double* out) {
  int G = d / 128;
  for (int j = j0; j < j0 + n; j++) {
    double val;
    if (tier == 3) {
      const uint8_t* p = rec + (int64_t)v * 2 * d + 2 * j;
      val = orc_f16_to_f32((uint16_t)(p[0] | (p[1] << 8)));
    } else {
      int64_t codes_bytes = (tier == 2) ? d : d / 2;
      const uint8_t* codes = rec + v * codes_bytes;
      const uint8_t* sc = rec + 3 * codes_bytes + (int64_t)v * 2 * G + 2 * (j / 128);
      double sv = orc_f16_to_f32((uint16_t)(sc[0] | (sc[1] << 8)));
      int q;
      if (tier == 2) {
        q = (int8_t)codes[j];
      } else {
        int nib = (j % 2 == 0) ? (codes[j / 2] & 0xf) : (codes[j / 2] >> 4);
        q = (nib >= 8) ? nib - 16 : nib;
      }
      val = q * sv;
    }
    out[j - j0] = val;
  }
}

/* Exact dequantized values (q * s, or the fp16 value) of one record. */
int orc_dequant_record(int d, int tier, const uint8_t* rec, double* gate, double* up,
                       double* down) {
  if (d <= 0 || d % 128 != 0 || tier < 1 || tier > 3) return -1;
  dequant_part(d, tier, rec, 0, 0, d, gate);
  dequant_part(d, tier, rec, 1, 0, d, up);
  dequant_part(d, tier, rec, 2, 0, d, down);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Low-rank predictor (Sec. 1 "Active Neuron Identification"; Sec. 5.2: the
 * predictor assigns a score to every neuron): z = A x, s = B z + bias, in
 * fp32 with one fixed evaluation order so scores are reproducible bit for bit:
 * chunks of 8 consecutive elements, chunk c feeds partial c % L with
 * L = min(64, largest power of two <= n/8), fmaf in ascending order, then
 * p[l] <- p[l] + p[l ^ off] for off = L/2 ... 1, result p[0].             */

static int canon_lanes(int n) {
  int chunks = n / 8, L = 1;
  while (L * 2 <= chunks && L < 64) L *= 2;
  return L;
}

static float canon_reduce(float* p, int L) {
  float t[64];
  for (int off = L / 2; off >= 1; off /= 2) {
    for (int l = 0; l < L; l++) t[l] = p[l] + p[l ^ off];
    for (int l = 0; l < L; l++) p[l] = t[l];
  }
  return p[0];
}

static float canon_dot_h_h(const uint16_t* a, const uint16_t* b, int n) {
  float p[64];
  int L = canon_lanes(n);
  for (int l = 0; l < 64; l++) p[l] = 0.0f;
  for (int c = 0; c < n / 8; c++)
    for (int e = 0; e < 8; e++)
      p[c % L] = fmaf(orc_f16_to_f32(a[8 * c + e]), orc_f16_to_f32(b[8 * c + e]), p[c % L]);
  return canon_reduce(p, L);
}

static float canon_dot_h_f(const uint16_t* a, const float* b, int n) {
  float p[64];
  int L = canon_lanes(n);
  for (int l = 0; l < 64; l++) p[l] = 0.0f;
  for (int c = 0; c < n / 8; c++)
    for (int e = 0; e < 8; e++)
      p[c % L] = fmaf(orc_f16_to_f32(a[8 * c + e]), b[8 * c + e], p[c % L]);
  return canon_reduce(p, L);
}

/* x [d] fp16 -> z [r] fp32, s [d_ff] fp32. bias may be NULL (no addition). */
int orc_predict(int d, int d_ff, int r, const uint16_t* A, const uint16_t* B, const float* bias,
                const uint16_t* x, float* z, float* s) {
  if (d <= 0 || d % 8 != 0 || r <= 0 || r % 8 != 0 || d_ff <= 0) return -1;
#pragma omp parallel for schedule(static)
  for (int j = 0; j < r; j++) z[j] = canon_dot_h_h(A + (int64_t)j * d, x, d);
#pragma omp parallel for schedule(static)
  for (int i = 0; i < d_ff; i++) {
    float v = canon_dot_h_f(B + (int64_t)i * r, z, r);
    if (bias) v = v + bias[i];
    s[i] = v;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Top-k and precision tiers (Sec. 5.2: the top-k scored neurons are active;
 * the higher the score, the higher the precision). Full sort by
 * (score descending, id ascending); scores compare as order-preserving keys
 * of their fp32 bits. Ranks [0,n16) FP16=3, [n16,n16+n8) INT8=2,
 * [n16+n8,k) INT4=1, others 0.                                             */

static uint32_t score_key(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

static const uint32_t* g_sort_keys;
static int cmp_rank(const void* pa, const void* pb) {
  int a = *(const int*)pa, b = *(const int*)pb;
  uint32_t ka = g_sort_keys[a], kb = g_sort_keys[b];
  if (ka != kb) return (ka > kb) ? -1 : 1;
  return (a < b) ? -1 : (a > b);
}

int orc_select_tiers(int d_ff, const float* s, int k, int n16, int n8, uint8_t* tier,
                     int32_t* ranked_ids) {
  if (d_ff <= 0 || k < 0 || k > d_ff || n16 < 0 || n8 < 0 || n16 + n8 > k) return -1;
  uint32_t* keys = (uint32_t*)malloc(sizeof(uint32_t) * d_ff);
  int* order = (int*)malloc(sizeof(int) * d_ff);
  for (int i = 0; i < d_ff; i++) { keys[i] = score_key(s[i]); order[i] = i; }
  g_sort_keys = keys;
  qsort(order, (size_t)d_ff, sizeof(int), cmp_rank);
  for (int rho = 0; rho < d_ff; rho++) {
    int i = order[rho];
    tier[i] = (rho < n16) ? 3 : (rho < n16 + n8) ? 2 : (rho < k) ? 1 : 0;
    if (ranked_ids && rho < k) ranked_ids[rho] = i;
  }
  free(keys);
  free(order);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Per-layer neuron slot cache (Sec. 5.3: one isolated cache unit per layer;
 * Sec. 1 and Sec. 6.4: LRU replacement of neurons in HBM). One step is
 * atomic: hits are decided against the cache before any eviction.
 *   tier of neuron i for the step = max over batch rows; R = {i : tier > 0}.
 *   For i in R, ascending, when i is resident at tier r and requested at t:
 *     policy 0 (exact tier): r == t -> HIT; otherwise REFILL in place at t.
 *     policy 1 (dominance): r >= t -> HIT, and the step uses i at tier r
 *       (the bytes in the slot are the record at tier r); r < t -> REFILL in
 *       place at t.
 *   Not resident -> NEW. Each NEW (ascending id) takes the untouched slot
 *   with the smallest (last_use, slot) found by a linear scan, evicting its
 *   neuron; when no untouched slot is left it is a BYPASS into staging slot
 *   C + j'. Every slot used by R gets last_use = step.
 * State arrays (in/out): slot_of [d_ff], slot_key/slot_tier/slot_last [C];
 * an empty slot has key -1 and last_use -1.
 * Outputs: counts [16]: 0 |R|, 1 HIT, 2 REFILL, 3 NEW, 4 BYPASS, 5 evictions,
 * 6 fills, 7..9 |R| at the step tier FP16 / INT8 / INT4, 10..12 fills by
 * tier FP16 / INT8 / INT4, the rest 0; the required list (ids, step tier,
 * hit code 0 NEW 1 HIT 2 REFILL 3 BYPASS, slot, row mask), the fill list
 * (every non-HIT in ascending id: id, tier, slot, and for a REFILL the tier
 * the slot held before the step, else 0) and the evicted ids in victim
 * order. Returns 0, -1 on bad arguments, -2 if the staging slots overflow. */

int orc_lru_plan(int d_ff, int C, int S, int B, const uint8_t* tier_map, int step, int policy,
                 int32_t* slot_of, int32_t* slot_key, uint8_t* slot_tier, int32_t* slot_last,
                 int32_t* counts, int32_t* req_ids, uint8_t* req_tier, uint8_t* req_hit,
                 int32_t* req_slot, uint32_t* req_mask, int32_t* fill_ids, uint8_t* fill_tier,
                 int32_t* fill_slot, uint8_t* fill_from, int32_t* evicted_ids) {
  if (d_ff <= 0 || C < 0 || S < 0 || B < 1 || B > 32 || policy < 0 || policy > 1) return -1;
  for (int c = 0; c < 16; c++) counts[c] = 0;
  uint8_t* touched = (uint8_t*)calloc((size_t)(C > 0 ? C : 1), 1);
  uint8_t* before = (uint8_t*)calloc((size_t)(d_ff > 0 ? d_ff : 1), 1); /* by position */
  int n = 0;
  for (int i = 0; i < d_ff; i++) {
    int t = 0;
    uint32_t m = 0;
    for (int b = 0; b < B; b++) {
      int tb = tier_map[(int64_t)b * d_ff + i];
      if (tb > 0) m |= 1u << b;
      if (tb > t) t = tb;
    }
    if (t == 0) continue;
    req_ids[n] = i;
    req_tier[n] = (uint8_t)t;
    req_mask[n] = m;
    n++;
  }
  counts[0] = n;
  /* hits and refills first: they pin their slots for this step */
  for (int p = 0; p < n; p++) {
    int i = req_ids[p], s = slot_of[i];
    if (s >= 0) {
      int r = slot_tier[s], t = req_tier[p];
      touched[s] = 1;
      before[p] = (uint8_t)r;
      if (r == t || (policy == 1 && r > t)) {
        req_hit[p] = 1;
        req_tier[p] = (uint8_t)r; /* the step uses the resident record */
        counts[1]++;
      } else {
        req_hit[p] = 2;
        counts[2]++;
        slot_tier[s] = (uint8_t)t;
      }
      req_slot[p] = s;
    } else {
      req_hit[p] = 0;
      req_slot[p] = -1;
    }
  }
  /* NEW neurons in ascending id take victims in (last_use, slot) order */
  int n_bypass = 0, n_evict = 0;
  for (int p = 0; p < n; p++) {
    if (req_hit[p] != 0) continue;
    int i = req_ids[p], v = -1;
    for (int s = 0; s < C; s++) {
      if (touched[s]) continue;
      if (v < 0 || slot_last[s] < slot_last[v]) v = s; /* ties keep the lower slot */
    }
    if (v < 0) {
      if (n_bypass >= S) { free(touched); free(before); return -2; } /* staging overflow */
      req_hit[p] = 3;
      req_slot[p] = C + n_bypass;
      n_bypass++;
      continue;
    }
    int old = slot_key[v];
    if (old >= 0) {
      slot_of[old] = -1;
      evicted_ids[n_evict++] = old;
    }
    touched[v] = 1;
    slot_key[v] = i;
    slot_tier[v] = req_tier[p];
    slot_of[i] = v;
    req_slot[p] = v;
    counts[3]++;
  }
  counts[4] = n_bypass;
  counts[5] = n_evict;
  for (int p = 0; p < n; p++)
    if (req_hit[p] != 3) slot_last[req_slot[p]] = step;
  int nf = 0;
  for (int p = 0; p < n; p++) {
    counts[7 + (3 - req_tier[p])]++;
    if (req_hit[p] == 1) continue;
    fill_ids[nf] = req_ids[p];
    fill_tier[nf] = req_tier[p];
    fill_slot[nf] = req_slot[p];
    fill_from[nf] = req_hit[p] == 2 ? before[p] : 0;
    counts[10 + (3 - req_tier[p])]++;
    nf++;
  }
  counts[6] = nf;
  free(touched);
  free(before);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Sparse mixed-precision SwiGLU FFN (Sec. 1 and Sec. 5.2: the FFN runs over
 * the active neurons only, each at its precision), in fp64 from the exact
 * dequantized weights: for batch row b,
 *   y_b = sum over listed neurons i with mask bit b of
 *         silu(<g_i, x_b>) * <u_i, x_b> * d_i,   silu(a) = a / (1 + e^-a).
 * ids [n] neuron ids, tiers [n], masks [n] (NULL = every row).
 * rec_fp16/int8/int4: record stores [d_ff][stride_t] (unused tiers may be NULL).
 * x [B][d] fp16; y [B][d] fp64.                                            */

int orc_sparse_ffn(int d, int B, int n, const int32_t* ids, const uint8_t* tiers,
                   const uint32_t* masks, const uint8_t* rec_fp16, int64_t stride_fp16,
                   const uint8_t* rec_int8, int64_t stride_int8, const uint8_t* rec_int4,
                   int64_t stride_int4, const uint16_t* x, double* y) {
  if (d <= 0 || d % 128 != 0 || B < 1 || n < 0) return -1;
  const uint8_t** recs = (const uint8_t**)malloc(sizeof(uint8_t*) * (n > 0 ? n : 1));
  for (int p = 0; p < n; p++) {
    int t = tiers[p];
    if (t == 3) recs[p] = rec_fp16 + (int64_t)ids[p] * stride_fp16;
    else if (t == 2) recs[p] = rec_int8 + (int64_t)ids[p] * stride_int8;
    else if (t == 1) recs[p] = rec_int4 + (int64_t)ids[p] * stride_int4;
    else { free(recs); return -1; }
  }
  double* xd = (double*)malloc(sizeof(double) * (size_t)B * d);
  for (int64_t j = 0; j < (int64_t)B * d; j++) xd[j] = orc_f16_to_f32(x[j]);
  /* h[p][b] = silu(<g_p, x_b>) * <u_p, x_b>, each dot product summed in
     ascending element order; 0 where row b does not select neuron p */
  double* h = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * B);
#pragma omp parallel
  {
    double* g = (double*)malloc(sizeof(double) * d);
    double* u = (double*)malloc(sizeof(double) * d);
#pragma omp for schedule(dynamic, 4)
    for (int p = 0; p < n; p++) {
      dequant_part(d, tiers[p], recs[p], 0, 0, d, g);
      dequant_part(d, tiers[p], recs[p], 1, 0, d, u);
      for (int b = 0; b < B; b++) {
        double hv = 0.0;
        if (!masks || ((masks[p] >> b) & 1u)) {
          double a = 0.0, c = 0.0;
          for (int j = 0; j < d; j++) {
            a += g[j] * xd[(int64_t)b * d + j];
            c += u[j] * xd[(int64_t)b * d + j];
          }
          hv = a / (1.0 + exp(-a)) * c;
        }
        h[(int64_t)p * B + b] = hv;
      }
    }
    free(g);
    free(u);
  }
  /* y_b[j] = sum over selected p, in ascending p, of h[p][b] * d_p[j], one
     quantization group of 128 output elements per task */
  int G = d / 128;
#pragma omp parallel
  {
    double dn[128];
#pragma omp for schedule(dynamic, 1)
    for (int gj = 0; gj < G; gj++) {
      for (int b = 0; b < B; b++)
        for (int j = 0; j < 128; j++) y[(int64_t)b * d + gj * 128 + j] = 0.0;
      for (int p = 0; p < n; p++) {
        dequant_part(d, tiers[p], recs[p], 2, gj * 128, 128, dn);
        for (int b = 0; b < B; b++) {
          if (masks && !((masks[p] >> b) & 1u)) continue;
          double hv = h[(int64_t)p * B + b];
          double* yb = y + (int64_t)b * d + gj * 128;
          for (int j = 0; j < 128; j++) yb[j] += hv * dn[j];
        }
      }
    }
  }
  free(h);
  free(xd);
  free(recs);
  return 0;
}

/* Dense SwiGLU FFN in fp64 (every neuron at fp16): the reference point the
 * sparse FFN must equal when k = d_ff and every neuron is FP16.            */
int orc_dense_ffn(int d, int d_ff, const uint16_t* w_gate, const uint16_t* w_up,
                  const uint16_t* w_down, const uint16_t* x, double* y) {
  if (d <= 0 || d_ff <= 0) return -1;
  double* xd = (double*)malloc(sizeof(double) * d);
  for (int j = 0; j < d; j++) { xd[j] = orc_f16_to_f32(x[j]); y[j] = 0.0; }
  for (int i = 0; i < d_ff; i++) {
    double a = 0.0, c = 0.0;
    for (int j = 0; j < d; j++) {
      a += orc_f16_to_f32(w_gate[(int64_t)i * d + j]) * xd[j];
      c += orc_f16_to_f32(w_up[(int64_t)i * d + j]) * xd[j];
    }
    double h = a / (1.0 + exp(-a)) * c;
    for (int j = 0; j < d; j++) y[j] += h * orc_f16_to_f32(w_down[(int64_t)j * d_ff + i]);
  }
  free(xd);
  return 0;
}

/* Array forms of the fp16 conversions (test convenience). */
void orc_f16_to_f32_n(const uint16_t* h, float* f, int64_t n) {
  for (int64_t i = 0; i < n; i++) f[i] = orc_f16_to_f32(h[i]);
}
void orc_f32_to_f16_n(const float* f, uint16_t* h, int64_t n) {
  for (int64_t i = 0; i < n; i++) h[i] = orc_f32_to_f16(f[i]);
}
