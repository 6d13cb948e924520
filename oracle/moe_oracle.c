/*
 * moe_oracle.c -- plain, slow CPU oracle for the fused block-scaled FP8
 * mixture-of-experts layer (the "Fused MoE" operator of the paper,
 * Section 3.1.1, stages (1)-(4)).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file: only tests/, __graft_entry__.smoke() and the cpu_baseline
 * leg of bench.py use it.  It shares no code, header, table or constant with
 * the HIP implementation.
 *
 * Every step follows the paper's order: (1) routing scores from a sigmoid,
 * group-limited top-k selection; (2) gathering the rows of each expert into a
 * contiguous FP8 layout with 128-element fp32 block scales; (3) the gated MLP:
 * FP8 block GEMM1 [rows,H]->[rows,2I], SwiGLU, re-quantisation, FP8 block
 * GEMM2 [rows,I]->[rows,H]; (4) scattering the expert outputs back to the
 * tokens, weighted by the routing scores.  Where the paper is silent the
 * reading used here is stated next to the code; all readings are collected in
 * the design notes of the repository.
 *
 * Precision: every GEMM and the combine are their plain definitions summed
 * in double (GEMM1 rounded once to fp32, SwiGLU's silu in double, the output
 * rounded once to bf16).  Routing follows one fixed fp32 sequence (the expert
 * choice is an integer decided by floating point, and the layer fixes the
 * sequence).  The re-quantised FP8 intermediate is also an integer decided by
 * floating point, but its inputs come from an FP8 block GEMM whose
 * accumulation the paper leaves to the matrix units: besides its own codes
 * the oracle states the set of codes any GEMM1 within a stated error model
 * admits (oracle_expert_admissible), and a device kernel is checked against
 * that set.
 *
 * The file also holds the oracle of the paper's DSA TopK Indexer (Section
 * 3.1.3), at its end.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fno-fast-math -shared -fPIC
 * (contraction must stay off: the fp32 routing sequence is a specification).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_BAD_ARG 1
#define ORACLE_NO_MEM 2

typedef struct {
  int32_t T, H, I;
  int32_t num_experts;       /* E_g, width of the router            */
  int32_t num_local_experts; /* E_l, experts whose weights are here */
  int32_t local_expert_offset;
  int32_t n_group, topk_group, top_k;
  float routed_scaling_factor;
} oracle_shape;

/* ------------------------------------------------------------------------ */
/* FP8 E4M3FN (OCP 8-bit floating point, E4M3 "FN": no infinities, a single  */
/* NaN mantissa pattern, max finite 448).  Stage (2) of Section 3.1.1 stores */
/* activations in FP8 with 128-element fp32 block scales.                     */
/* ------------------------------------------------------------------------ */

/* Decode one code from its bit fields: sign, 4-bit exponent (bias 7),
 * 3-bit mantissa; exponent field 0 is subnormal (m * 2^-9); S.1111.111 is NaN. */
double oracle_e4m3_decode(uint8_t q) {
  int sign = (q >> 7) & 1;
  int ef = (q >> 3) & 0xF;
  int mf = q & 0x7;
  double v;
  if (ef == 0xF && mf == 0x7) return NAN;
  if (ef == 0)
    v = ldexp((double)mf, -9);
  else
    v = ldexp(1.0 + mf / 8.0, ef - 7);
  return sign ? -v : v;
}

/* Encode an fp32 value: round to nearest, ties to even mantissa, saturating
 * to +-448 (the re-quantised values never exceed 448 by more than a rounding
 * error; saturation is the reading taken for that case).  NaN -> 0x7F. */
uint8_t oracle_e4m3_encode(float v) {
  uint8_t s;
  double a, quantum, m, r;
  int e, E;
  if (isnan(v)) return 0x7F;
  s = signbit(v) ? 0x80 : 0x00;
  a = fabs((double)v);
  if (a >= 448.0) return (uint8_t)(s | 0x7E);
  if (a == 0.0) return s;
  frexp(a, &e);           /* a in [2^(e-1), 2^e) */
  E = e - 1;
  if (E < -6) E = -6;     /* subnormal binade shares the quantum 2^-9 */
  quantum = ldexp(1.0, E - 3);
  m = nearbyint(a / quantum); /* exact division by a power of two; RNE */
  r = m * quantum;
  if (r == 0.0) return s;
  frexp(r, &e);           /* re-derive the binade: rounding may carry up */
  E = e - 1;
  if (E < -6) {
    return (uint8_t)(s | (int)(r / ldexp(1.0, -9)));
  }
  {
    int mant = (int)(r / ldexp(1.0, E - 3)) - 8;
    return (uint8_t)(s | ((E + 7) << 3) | mant);
  }
}

void oracle_e4m3_encode_array(const float *x, uint8_t *q, int64_t n) {
  int64_t i;
#pragma omp parallel for schedule(static)
  for (i = 0; i < n; ++i) q[i] = oracle_e4m3_encode(x[i]);
}

/* bf16 (8 significant bits, fp32 exponent range) from a double, rounded once
 * to nearest even; the combine of stage (4) writes bf16. */
uint16_t oracle_bf16_from_double(double v) {
  uint16_t sign;
  double a, m, r;
  int e, qexp;
  float f;
  uint32_t bits;
  if (isnan(v)) return 0x7FC0;
  sign = signbit(v) ? 0x8000 : 0;
  a = fabs(v);
  if (a == 0.0) return sign;
  frexp(a, &e);           /* a in [2^(e-1), 2^e): quantum 2^(e-8) */
  qexp = e - 8;
  if (qexp < -133) qexp = -133; /* bf16 subnormal quantum */
  m = nearbyint(ldexp(a, -qexp));
  r = ldexp(m, qexp);
  f = (float)r;           /* exact (or +inf past the bf16 range) */
  memcpy(&bits, &f, 4);
  return (uint16_t)(sign | (bits >> 16));
}

/* ------------------------------------------------------------------------ */
/* Routing sigmoid.  Stage (1) applies a sigmoid to the router logits.  Two  */
/* faithful fp32 sigmoids that differ in the last bit can pick different     */
/* experts when two keys are within an ulp, so the layer fixes one fp32      */
/* operation sequence (Cody-Waite reduction of exp, degree-7 Taylor          */
/* polynomial in Horner form with fused multiply-adds, IEEE division).  The  */
/* constants come from ln 2, log2 e and 1/k!, rounded to fp32.               */
/* ------------------------------------------------------------------------ */
float oracle_sigmoid(float x) {
  const float log2e = 1.44269502f;          /* log2(e) rounded to fp32      */
  const float ln2_hi = 0.693145751953125f;  /* ln 2 with 12 low bits clear  */
  const float ln2_lo = 1.42860677e-6f;      /* fp32(ln 2 - ln2_hi)          */
  float z, n, r, p, e;
  if (x < -80.0f) x = -80.0f;
  if (x > 80.0f) x = 80.0f;
  z = -x;                                   /* sigma(x) = 1 / (1 + e^z) */
  n = rintf(z * log2e);                     /* nearest, ties to even     */
  r = fmaf(-n, ln2_hi, z);
  r = fmaf(-n, ln2_lo, r);
  p = 1.0f / 5040.0f;                       /* 1/7! */
  p = fmaf(p, r, 1.0f / 720.0f);            /* 1/6! */
  p = fmaf(p, r, 1.0f / 120.0f);            /* 1/5! */
  p = fmaf(p, r, 1.0f / 24.0f);             /* 1/4! */
  p = fmaf(p, r, 1.0f / 6.0f);              /* 1/3! */
  p = fmaf(p, r, 0.5f);                     /* 1/2! */
  p = fmaf(p, r, 1.0f);
  p = fmaf(p, r, 1.0f);
  e = ldexpf(p, (int)n);
  return 1.0f / (1.0f + e);
}

void oracle_sigmoid_array(const float *x, float *y, int64_t n) {
  int64_t i;
#pragma omp parallel for schedule(static)
  for (i = 0; i < n; ++i) y[i] = oracle_sigmoid(x[i]);
}

/* ------------------------------------------------------------------------ */
/* Stage (1): DeepSeek-V3 group-limited routing for one token.               */
/*   s_e   = sigmoid(logit_e)                       (fp32)                   */
/*   key_e = s_e + bias_e                           (fp32; selection only)  */
/*   gs_g  = sum of the two largest keys of group g (fp32)                   */
/*   keep the topk_group groups of largest gs, then the top_k experts of     */
/*   largest key inside them; order: larger value first, ties -> lower index */
/*   w_j   = s_{id_j} / (sum over the k selected s) * routed_scaling_factor  */
/*           (sum in selection order, over all k, local or not)              */
/* ------------------------------------------------------------------------ */
static int beats(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

static void route_token(const oracle_shape *s, const float *logit,
                        const float *bias, int32_t *ids, float *w) {
  int E = s->num_experts, G = s->n_group, gsz = E / G;
  float *sc = (float *)malloc(sizeof(float) * E);
  float *key = (float *)malloc(sizeof(float) * E);
  float *gs = (float *)malloc(sizeof(float) * G);
  char *gkeep = (char *)calloc(G, 1);
  char *taken = (char *)calloc(E, 1);
  int e, g, j, r;
  float sum;

  for (e = 0; e < E; ++e) {
    sc[e] = oracle_sigmoid(logit[e]);
    key[e] = sc[e] + bias[e];
  }
  for (g = 0; g < G; ++g) {
    int b1 = -1, b2 = -1;
    for (e = g * gsz; e < (g + 1) * gsz; ++e) {
      if (b1 < 0 || beats(key[e], e, key[b1], b1)) {
        b2 = b1;
        b1 = e;
      } else if (b2 < 0 || beats(key[e], e, key[b2], b2)) {
        b2 = e;
      }
    }
    gs[g] = key[b1] + key[b2];
  }
  for (r = 0; r < s->topk_group; ++r) {
    int best = -1;
    for (g = 0; g < G; ++g)
      if (!gkeep[g] && (best < 0 || beats(gs[g], g, gs[best], best))) best = g;
    gkeep[best] = 1;
  }
  for (j = 0; j < s->top_k; ++j) {
    int best = -1;
    for (e = 0; e < E; ++e) {
      if (!gkeep[e / gsz] || taken[e]) continue;
      if (best < 0 || beats(key[e], e, key[best], best)) best = e;
    }
    taken[best] = 1;
    ids[j] = best;
  }
  sum = 0.0f;
  for (j = 0; j < s->top_k; ++j) sum += sc[ids[j]];
  for (j = 0; j < s->top_k; ++j)
    w[j] = (sc[ids[j]] / sum) * s->routed_scaling_factor;

  free(sc);
  free(key);
  free(gs);
  free(gkeep);
  free(taken);
}

int oracle_check_shape(const oracle_shape *s) {
  if (!s) return ORACLE_BAD_ARG;
  if (s->T < 0 || s->H <= 0 || s->I <= 0) return ORACLE_BAD_ARG;
  if (s->H % 128 || s->I % 128) return ORACLE_BAD_ARG;
  if (s->num_experts <= 0 || s->n_group <= 0) return ORACLE_BAD_ARG;
  if (s->num_experts % s->n_group) return ORACLE_BAD_ARG;
  if (s->num_experts / s->n_group < 2) return ORACLE_BAD_ARG;
  if (s->topk_group <= 0 || s->topk_group > s->n_group) return ORACLE_BAD_ARG;
  if (s->top_k <= 0 ||
      s->top_k > s->topk_group * (s->num_experts / s->n_group))
    return ORACLE_BAD_ARG;
  if (s->num_local_experts <= 0 || s->local_expert_offset < 0 ||
      s->local_expert_offset + s->num_local_experts > s->num_experts)
    return ORACLE_BAD_ARG;
  return ORACLE_OK;
}

int oracle_route(const oracle_shape *s, const float *logits, const float *bias,
                 int32_t *topk_ids, float *topk_w) {
  int t;
  if (oracle_check_shape(s)) return ORACLE_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 16)
  for (t = 0; t < s->T; ++t)
    route_token(s, logits + (int64_t)t * s->num_experts, bias,
                topk_ids + (int64_t)t * s->top_k, topk_w + (int64_t)t * s->top_k);
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Stage (1)'s router projection: the routing scores start from a linear     */
/* projection of the token's hidden state onto one weight row per expert.   */
/* Here the hidden state is the FP8 row with its 1x128 block scales (the     */
/* input of stage (2)), the router weight is fp32 [E_g, H], and the logits   */
/* are fp32.  The paper does not fix the projection's precision; since the   */
/* logits decide the expert choice, the layer fixes one fp32 sequence:      */
/*   p_kb    = fused multiply-add chain over the 128 elements of block kb,   */
/*             ascending, from 0:  p = fmaf(dec(q[h]), W[e][h], p)           */
/*             (dec(q) is exact in fp32; the block scale is not applied)    */
/*   logit_e = fused multiply-add chain over the blocks, ascending, from 0:  */
/*             acc = fmaf(scale[kb], p_kb, acc)                              */
/* Reading: the logits are the dequantised hidden row times the weight row, */
/* accumulated blockwise in fp32 (error bound: (128 + H/128) u sum |x w|).  */
/* ------------------------------------------------------------------------ */
int oracle_router_logits(const oracle_shape *s, const uint8_t *hidden,
                         const float *hidden_scale, const float *weight,
                         float *logits) {
  int64_t t;
  int HB;
  if (oracle_check_shape(s)) return ORACLE_BAD_ARG;
  HB = s->H / 128;
#pragma omp parallel for schedule(dynamic, 1)
  for (t = 0; t < s->T; ++t) {
    const uint8_t *q = hidden + t * s->H;
    const float *sc = hidden_scale + t * HB;
    int e, kb, i;
    for (e = 0; e < s->num_experts; ++e) {
      const float *w = weight + (int64_t)e * s->H;
      float acc = 0.0f;
      for (kb = 0; kb < HB; ++kb) {
        float p = 0.0f;
        for (i = 0; i < 128; ++i) {
          int h = kb * 128 + i;
          p = fmaf((float)oracle_e4m3_decode(q[h]), w[h], p);
        }
        acc = fmaf(sc[kb], p, acc);
      }
      logits[t * s->num_experts + e] = acc;
    }
  }
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Stage (2) bookkeeping: the (token, slot) pairs whose expert is resident   */
/* are grouped by local expert into one contiguous layout.  Order inside an  */
/* expert: ascending token (a token holds an expert at most once).           */
/*   expert_offsets[e] = first row of local expert e, [E_l] = P              */
/*   perm_token[row]   = token of that row                                   */
/*   pair_row[t*k+j]   = row of pair (t, j), -1 when its expert is remote    */
/* ------------------------------------------------------------------------ */
int oracle_permute(const oracle_shape *s, const int32_t *topk_ids,
                   int32_t *expert_offsets, int32_t *perm_token,
                   int32_t *pair_row) {
  int64_t pos = 0, p, npairs;
  int e, t, j, k;
  if (oracle_check_shape(s)) return ORACLE_BAD_ARG;
  k = s->top_k;
  npairs = (int64_t)s->T * k;
  for (p = 0; p < npairs; ++p) pair_row[p] = -1;
  for (e = 0; e < s->num_local_experts; ++e) {
    int gid = s->local_expert_offset + e;
    expert_offsets[e] = (int32_t)pos;
    for (t = 0; t < s->T; ++t)
      for (j = 0; j < k; ++j)
        if (topk_ids[(int64_t)t * k + j] == gid) {
          perm_token[pos] = t;
          pair_row[(int64_t)t * k + j] = (int32_t)pos;
          ++pos;
        }
  }
  expert_offsets[s->num_local_experts] = (int32_t)pos;
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Decoded e4m3 values as a 256-entry table (each entry from the bit-field   */
/* decoder above), so the GEMM loops below read one double per code.         */
/* Filled once, before any parallel region, by every entry point using it.   */
/* ------------------------------------------------------------------------ */
static double dec_tab[256];
static int dec_tab_ready = 0;

static void dec_table_init(void) {
  int c;
  if (dec_tab_ready) return;
  for (c = 0; c < 256; ++c) dec_tab[c] = oracle_e4m3_decode((uint8_t)c);
  dec_tab_ready = 1;
}

/* Unbiased exponent of an e4m3 code's exponent field (-6 for field 0, the   */
/* subnormal binade): a code's value is a multiple of 2^(exponent - 3).      */
static int e4m3_exponent(uint8_t q) {
  int ef = (q >> 3) & 0xF;
  return ef == 0 ? -6 : ef - 7;
}

/* SwiGLU of stage (3) from its definition: silu(g) * u with                 */
/* silu(z) = z / (1 + e^-z) evaluated in double, the product rounded once    */
/* to fp32.                                                                  */
static double silu_d(double z) { return z / (1.0 + exp(-z)); }

float oracle_swiglu(float g, float u) { return (float)(silu_d((double)g) * (double)u); }

/* GEMM1 of one token row against one expert, from its definition: for each  */
/* output row n, the exact products of the dequantised operands summed in    */
/* double (x = dec(hidden) * hidden_scale and w = dec(w13) * w13_scale are   */
/* exact in double).  Optionally also, per n, the two sums the admissible-   */
/* set bound needs: abs_sum[n] = sum |x w| and blk_sum[n] = sum over blocks  */
/* kb of |sa sw| 2^(E_kb - 6), E_kb the largest exponent sum                 */
/* exp(a_k) + exp(w_k) over the block's 128 code pairs.                      */
static void gemm1_row(int32_t H, int32_t n2, const uint8_t *hidden_row,
                      const float *hidden_scale_row, const uint8_t *w13,
                      const float *w13_scale, double *g, double *abs_sum,
                      double *blk_sum) {
  int HB = H / 128, n, kb, k;
  for (n = 0; n < n2; ++n) {
    const uint8_t *wr = w13 + (int64_t)n * H;
    const float *sr = w13_scale + (int64_t)(n / 128) * HB;
    double acc = 0.0, aabs = 0.0, ablk = 0.0;
    for (kb = 0; kb < HB; ++kb) {
      double sa = hidden_scale_row[kb], sw = sr[kb];
      for (k = kb * 128; k < kb * 128 + 128; ++k)
        acc += (dec_tab[hidden_row[k]] * sa) * (dec_tab[wr[k]] * sw);
      if (abs_sum) {
        int E = -1000;
        double pabs = 0.0;
        for (k = kb * 128; k < kb * 128 + 128; ++k) {
          int ek = e4m3_exponent(hidden_row[k]) + e4m3_exponent(wr[k]);
          if (ek > E) E = ek;
          pabs += fabs(dec_tab[hidden_row[k]] * dec_tab[wr[k]]);
        }
        aabs += fabs(sa * sw) * pabs;
        ablk += fabs(sa * sw) * ldexp(1.0, E - 6);
      }
    }
    g[n] = acc;
    if (abs_sum) abs_sum[n] = aabs;
    if (blk_sum) blk_sum[n] = ablk;
  }
}

/* Re-quantisation of one row of SwiGLU outputs, per 1x128 block:           */
/*   amax = max |a| (fp32); scale = amax / 448 (fp32 division);              */
/*   q = e4m3(a / scale) (fp32 division, round to nearest even, saturating); */
/*   an all-zero block gets scale 1 and codes 0.                             */
static void requant_row(int32_t I, const float *a, uint8_t *q, float *qs) {
  int b, i;
  for (b = 0; b < I / 128; ++b) {
    float amax = 0.0f, scale;
    for (i = b * 128; i < (b + 1) * 128; ++i) {
      float m = fabsf(a[i]);
      if (m > amax) amax = m;
    }
    scale = (amax == 0.0f) ? 1.0f : amax / 448.0f;
    qs[b] = scale;
    for (i = b * 128; i < (b + 1) * 128; ++i)
      q[i] = (amax == 0.0f) ? 0 : oracle_e4m3_encode(a[i] / scale);
  }
}

/* ------------------------------------------------------------------------ */
/* Stage (3): the gated MLP of one expert applied to one token row, from the */
/* plain definition of each step (double wherever floating point decides no  */
/* integer):                                                                 */
/*   g[n] = fp32( sum_h x[h] w13[n,h] )  in double;  rows [0,I) gate,        */
/*          [I,2I) up                                                         */
/*   a[i] = fp32( silu(g[i]) * g[I+i] ),  silu in double                     */
/*   (q, scale) = the 1x128 re-quantisation of a (requant_row above)         */
/*   y[n] = sum_i dec(q[i]) scale[i/128] dec(w2[n,i]) w2_scale[n/128,i/128]  */
/*          in double                                                         */
/* Optional outputs: g (fp32, 2I), q (I codes), qscale (I/128).              */
/* ------------------------------------------------------------------------ */
void oracle_expert_ffn(int32_t H, int32_t I, const uint8_t *hidden_row,
                       const float *hidden_scale_row, const uint8_t *w13,
                       const float *w13_scale, const uint8_t *w2,
                       const float *w2_scale, double *y, float *g_out,
                       uint8_t *q_out, float *qscale_out) {
  int IB = I / 128;
  double *gd = (double *)malloc(sizeof(double) * 2 * I);
  float *g = (float *)malloc(sizeof(float) * 2 * I);
  float *a = (float *)malloc(sizeof(float) * I);
  uint8_t *q = (uint8_t *)malloc(I);
  float *qs = (float *)malloc(sizeof(float) * IB);
  double *aq = (double *)malloc(sizeof(double) * I);
  int n, i;

  dec_table_init();
  gemm1_row(H, 2 * I, hidden_row, hidden_scale_row, w13, w13_scale, gd, NULL, NULL);
  for (n = 0; n < 2 * I; ++n) g[n] = (float)gd[n];
  for (i = 0; i < I; ++i) a[i] = oracle_swiglu(g[i], g[I + i]);
  requant_row(I, a, q, qs);
  for (i = 0; i < I; ++i) aq[i] = dec_tab[q[i]] * (double)qs[i / 128];
  for (n = 0; n < H; ++n) {
    const uint8_t *wr = w2 + (int64_t)n * I;
    const float *sr = w2_scale + (int64_t)(n / 128) * IB;
    double acc = 0.0;
    for (i = 0; i < I; ++i) acc += aq[i] * (dec_tab[wr[i]] * (double)sr[i / 128]);
    y[n] = acc;
  }
  if (g_out) memcpy(g_out, g, sizeof(float) * 2 * I);
  if (q_out) memcpy(q_out, q, I);
  if (qscale_out) memcpy(qscale_out, qs, sizeof(float) * IB);
  free(gd);
  free(g);
  free(a);
  free(q);
  free(qs);
  free(aq);
}

/* ------------------------------------------------------------------------ */
/* The admissible re-quantised intermediate of one (token, expert) pair.     */
/* Stage (3) turns GEMM1's output into integers (the FP8 codes), and GEMM1   */
/* is an FP8 block GEMM whose accumulation precision the paper leaves to the */
/* matrix units; a device kernel's codes are therefore not compared for      */
/* equality but checked for membership in the set that every GEMM1 within    */
/* the following error model produces:                                       */
/*  (i)  the 128 exact e4m3 products p_k of a K block are accumulated at a   */
/*       resolution no coarser than 2^(E_kb - 13), E_kb the largest exponent */
/*       sum exp(a_k) + exp(w_k) of the block (each product is a multiple of */
/*       2^(exp(a)+exp(w)-6) below 2^(exp(a)+exp(w)+2): 13 fraction bits of */
/*       the block's leading product exponent), with fp32 rounding of        */
/*       partial sums:  |t' - t| <= beta_kb = 2^(E_kb-6) + 2^-19 sum|p_k|;   */
/*  (ii) the block sums are scaled by fp32(sa*sw) and added in fp32, in any  */
/*       order (a split K included): at most gamma(nb+2) (sum|x w| + sum    */
/*       |sa sw| beta_kb) more, gamma(m) = m u / (1 - m u), u = 2^-24;       */
/*  (iii) SwiGLU is evaluated in fp32 with relative error at most 8 u (plus  */
/*       1e-30 absolute for inputs whose sigmoid underflows);                 */
/*  (iv) amax, scale = amax/448 and the codes then follow exactly (fp32      */
/*       division, nearest-even, saturating), the ratio allowed 2 ulps.       */
/* So g' lies in [g - dg, g + dg], dg = sum|sa sw| beta_kb + (i)'s and (ii)'s */
/* fp32 terms (+ 2^-50 sum|x w| for the double sum itself); a' in the range  */
/* of silu(g')u' over that box, widened by (iii); the block's scale in        */
/* [fp32(amax_lo/448), fp32(amax_hi/448)]; each code's value in               */
/* [dec(e4m3(r_lo)), dec(e4m3(r_hi))] over the extreme ratios a'/scale'.     */
/* An all-zero block (scale 1, codes 0) is admissible when amax_lo = 0.      */
/* Outputs per pair: v_lo/v_hi [I] (admissible code values), s_lo/s_hi [I/128]*/
/* (admissible scales), zero_ok [I/128], and the nominal codes/scales of     */
/* oracle_expert_ffn (q [I], qs [I/128]).                                    */
/* ------------------------------------------------------------------------ */
static const double kSiluArgMin = -1.2784645427610738; /* root of silu' */

static void silu_range(double lo, double hi, double *mn, double *mx) {
  double a = silu_d(lo), b = silu_d(hi);
  *mn = a < b ? a : b;
  *mx = a > b ? a : b;
  if (lo <= kSiluArgMin && kSiluArgMin <= hi) {
    double m = silu_d(kSiluArgMin);
    if (m < *mn) *mn = m;
  }
}

static float next_down(float x, int k) {
  while (k--) x = nextafterf(x, -INFINITY);
  return x;
}
static float next_up(float x, int k) {
  while (k--) x = nextafterf(x, INFINITY);
  return x;
}

void oracle_expert_admissible(int32_t H, int32_t I, const uint8_t *hidden_row,
                              const float *hidden_scale_row, const uint8_t *w13,
                              const float *w13_scale, uint8_t *q, float *qs,
                              float *v_lo, float *v_hi, float *s_lo, float *s_hi,
                              uint8_t *zero_ok) {
  const double u = ldexp(1.0, -24);
  const int HB = H / 128, IB = I / 128;
  const double gam = (HB + 2) * u / (1.0 - (HB + 2) * u);
  double *gd = (double *)malloc(sizeof(double) * 2 * I);
  double *sabs = (double *)malloc(sizeof(double) * 2 * I);
  double *sblk = (double *)malloc(sizeof(double) * 2 * I);
  double *dg = (double *)malloc(sizeof(double) * 2 * I);
  float *a = (float *)malloc(sizeof(float) * I);
  double *alo = (double *)malloc(sizeof(double) * I);
  double *ahi = (double *)malloc(sizeof(double) * I);
  int n, i, b;

  dec_table_init();
  gemm1_row(H, 2 * I, hidden_row, hidden_scale_row, w13, w13_scale, gd, sabs, sblk);
  for (n = 0; n < 2 * I; ++n) {
    double beta = sblk[n] + ldexp(1.0, -19) * sabs[n]; /* (i), summed over kb */
    dg[n] = beta + gam * (sabs[n] + beta) + ldexp(1.0, -50) * sabs[n];
  }
  /* the nominal intermediate (the oracle's own codes) */
  for (i = 0; i < I; ++i) a[i] = oracle_swiglu((float)gd[i], (float)gd[I + i]);
  requant_row(I, a, q, qs);
  /* (iii): the range of silu(g') u' over the box, widened */
  for (i = 0; i < I; ++i) {
    double smn, smx, ulo = gd[I + i] - dg[I + i], uhi = gd[I + i] + dg[I + i];
    double c[4], lo, hi, m;
    int k;
    silu_range(gd[i] - dg[i], gd[i] + dg[i], &smn, &smx);
    c[0] = smn * ulo;
    c[1] = smn * uhi;
    c[2] = smx * ulo;
    c[3] = smx * uhi;
    lo = hi = c[0];
    for (k = 1; k < 4; ++k) {
      if (c[k] < lo) lo = c[k];
      if (c[k] > hi) hi = c[k];
    }
    m = fabs(lo) > fabs(hi) ? fabs(lo) : fabs(hi);
    alo[i] = lo - 8 * u * m - 1e-30;
    ahi[i] = hi + 8 * u * m + 1e-30;
  }
  /* (iv) per block: admissible amax and scale, then each code's range */
  for (b = 0; b < IB; ++b) {
    double mlo = 0.0, mhi = 0.0;
    float sl, sh, flo, fhi;
    for (i = b * 128; i < (b + 1) * 128; ++i) {
      double mn = (alo[i] <= 0.0 && ahi[i] >= 0.0) ? 0.0
                  : (fabs(alo[i]) < fabs(ahi[i]) ? fabs(alo[i]) : fabs(ahi[i]));
      double mx = fabs(alo[i]) > fabs(ahi[i]) ? fabs(alo[i]) : fabs(ahi[i]);
      if (mn > mlo) mlo = mn;
      if (mx > mhi) mhi = mx;
    }
    /* the kernel's amax is the largest of its fp32 values: an fp32 number   */
    flo = next_down((float)mlo, 1);
    if (flo < 0.0f) flo = 0.0f;
    fhi = next_up((float)mhi, 1);
    zero_ok[b] = flo == 0.0f;
    sl = flo / 448.0f;
    sh = fhi / 448.0f;
    if (sl == 0.0f) sl = nextafterf(0.0f, 1.0f); /* a nonzero amax's scale */
    s_lo[b] = sl;
    s_hi[b] = sh;
    for (i = b * 128; i < (b + 1) * 128; ++i) {
      float lo = (float)alo[i], hi = (float)ahi[i], rlo, rhi;
      lo = next_down(lo, 1);
      hi = next_up(hi, 1);
      rlo = lo >= 0.0f ? lo / sh : lo / sl;
      rhi = hi >= 0.0f ? hi / sl : hi / sh;
      rlo = next_down(rlo, 2);
      rhi = next_up(rhi, 2);
      v_lo[i] = (float)dec_tab[oracle_e4m3_encode(rlo)];
      v_hi[i] = (float)dec_tab[oracle_e4m3_encode(rhi)];
      if (zero_ok[b]) {
        if (v_lo[i] > 0.0f) v_lo[i] = 0.0f;
        if (v_hi[i] < 0.0f) v_hi[i] = 0.0f;
      }
    }
  }
  free(gd);
  free(sabs);
  free(sblk);
  free(dg);
  free(a);
  free(alo);
  free(ahi);
}

/* oracle_expert_admissible for a list of n (token, local expert) pairs, in  */
/* parallel; outputs are [n, I] and [n, I/128] arrays in list order.         */
int oracle_admissible_batch(const oracle_shape *s, const uint8_t *hidden,
                            const float *hidden_scale, const uint8_t *const *w13,
                            const float *const *w13_scale, int32_t n,
                            const int32_t *tokens, const int32_t *experts,
                            uint8_t *q, float *qs, float *v_lo, float *v_hi,
                            float *s_lo, float *s_hi, uint8_t *zero_ok) {
  int32_t p;
  int H = s->H, I = s->I, HB, IB, bad = 0;
  if (oracle_check_shape(s) || n < 0) return ORACLE_BAD_ARG;
  HB = H / 128;
  IB = I / 128;
  for (p = 0; p < n; ++p) {
    int e = experts[p];
    if (tokens[p] < 0 || tokens[p] >= s->T || e < 0 || e >= s->num_local_experts ||
        !w13[e] || !w13_scale[e])
      bad = 1;
  }
  if (bad) return ORACLE_BAD_ARG;
  dec_table_init();
#pragma omp parallel for schedule(dynamic, 1)
  for (p = 0; p < n; ++p) {
    int e = experts[p];
    int64_t t = tokens[p];
    oracle_expert_admissible(H, I, hidden + t * H, hidden_scale + t * HB, w13[e], w13_scale[e],
                             q + (int64_t)p * I, qs + (int64_t)p * IB, v_lo + (int64_t)p * I,
                             v_hi + (int64_t)p * I, s_lo + (int64_t)p * IB,
                             s_hi + (int64_t)p * IB, zero_ok + (int64_t)p * IB);
  }
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Stage (3)'s GEMM2 and stage (4)'s combine from a given re-quantised       */
/* intermediate: act [P, I] e4m3 with act_scale [P, I/128], rows in the      */
/* permuted order of oracle_permute (expert_offsets, pair_row), for the      */
/* listed tokens:                                                            */
/*   out[r, n] = bf16( sum over local slots j of token_list[r], in slot      */
/*               order, of w_j * y_j[n] ),                                    */
/*   y_j[n] = sum_i dec(act[row,i]) act_scale[row,i/128] dec(w2[e,n,i])      */
/*            w2_scale[e,n/128,i/128]   (double), row = pair_row[t,j]         */
/* ------------------------------------------------------------------------ */
int oracle_combine_from_act(const oracle_shape *s, const uint8_t *act,
                            const float *act_scale, const uint8_t *const *w2,
                            const float *const *w2_scale, const int32_t *expert_offsets,
                            const int32_t *pair_row, const float *topk_w,
                            const int32_t *token_list, int32_t n_tokens, uint16_t *out) {
  int H = s->H, I = s->I, k = s->top_k, IB, El = s->num_local_experts;
  int32_t r;
  if (oracle_check_shape(s) || n_tokens < 0) return ORACLE_BAD_ARG;
  IB = I / 128;
  for (r = 0; r < n_tokens; ++r)
    if (token_list[r] < 0 || token_list[r] >= s->T) return ORACLE_BAD_ARG;
  dec_table_init();
#pragma omp parallel for schedule(dynamic, 1)
  for (r = 0; r < n_tokens; ++r) {
    int64_t t = token_list[r];
    double *acc = (double *)calloc(H, sizeof(double));
    double *aq = (double *)malloc(sizeof(double) * I);
    int j, n, i;
    for (j = 0; j < k; ++j) {
      int row = pair_row[t * k + j], e = 0;
      double wj;
      if (row < 0) continue;
      while (e + 1 < El && expert_offsets[e + 1] <= row) ++e;
      wj = (double)topk_w[t * k + j];
      for (i = 0; i < I; ++i)
        aq[i] = dec_tab[act[(int64_t)row * I + i]] * (double)act_scale[(int64_t)row * IB + i / 128];
      for (n = 0; n < H; ++n) {
        const uint8_t *wr = w2[e] + (int64_t)n * I;
        const float *sr = w2_scale[e] + (int64_t)(n / 128) * IB;
        double y = 0.0;
        for (i = 0; i < I; ++i) y += aq[i] * (dec_tab[wr[i]] * (double)sr[i / 128]);
        acc[n] += wj * y;
      }
    }
    for (n = 0; n < H; ++n) out[(int64_t)r * H + n] = oracle_bf16_from_double(acc[n]);
    free(acc);
    free(aq);
  }
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* The whole layer for a list of tokens (stages 1-4).  Tokens are            */
/* independent, so any subset of rows can be computed exactly.               */
/*   out[r, n] = bf16( sum over local slots j of token_list[r], in slot      */
/*               order, of w_j * y_j[n] )   (double sum, one rounding)       */
/* A token with no resident expert gets +0.  Weight pointers are per local   */
/* expert; an expert no listed token uses may be NULL.                       */
/* ------------------------------------------------------------------------ */
int oracle_forward(const oracle_shape *s, const uint8_t *hidden,
                   const float *hidden_scale, const float *logits,
                   const float *bias, const uint8_t *const *w13,
                   const float *const *w13_scale, const uint8_t *const *w2,
                   const float *const *w2_scale, const int32_t *token_list,
                   int32_t n_tokens, uint16_t *out, int32_t *ids_out,
                   float *w_out) {
  int H = s->H, I = s->I, k = s->top_k, HB;
  int32_t *ids, *pr_t, *pr_e, np = 0;
  float *w;
  double *acc, *ys;
  int r, j, p, n, bad = 0;
  if (oracle_check_shape(s)) return ORACLE_BAD_ARG;
  if (n_tokens < 0 || (n_tokens > 0 && !token_list)) return ORACLE_BAD_ARG;
  dec_table_init();
  HB = H / 128;
  ids = (int32_t *)malloc(sizeof(int32_t) * ((size_t)n_tokens * k + 1));
  w = (float *)malloc(sizeof(float) * ((size_t)n_tokens * k + 1));
  pr_t = (int32_t *)malloc(sizeof(int32_t) * ((size_t)n_tokens * k + 1));
  pr_e = (int32_t *)malloc(sizeof(int32_t) * ((size_t)n_tokens * k + 1));
  if (!ids || !w || !pr_t || !pr_e) return ORACLE_NO_MEM;

  /* (1) routing */
  for (r = 0; r < n_tokens; ++r) {
    int t = token_list[r];
    if (t < 0 || t >= s->T) return ORACLE_BAD_ARG;
    route_token(s, logits + (int64_t)t * s->num_experts, bias,
                ids + (int64_t)r * k, w + (int64_t)r * k);
  }
  /* (2) the resident (token, slot) pairs */
  for (r = 0; r < n_tokens; ++r)
    for (j = 0; j < k; ++j) {
      int le = ids[r * k + j] - s->local_expert_offset;
      if (le >= 0 && le < s->num_local_experts) {
        pr_t[np] = r * k + j;
        pr_e[np] = le;
        ++np;
      }
    }
  for (p = 0; p < np; ++p) {
    int le = pr_e[p];
    if (!w13[le] || !w13_scale[le] || !w2[le] || !w2_scale[le]) bad = 1;
  }
  if (bad) return ORACLE_BAD_ARG;

  /* (3) the gated MLP of every resident pair */
  ys = (double *)malloc(sizeof(double) * ((size_t)np * H + 1));
  if (!ys) return ORACLE_NO_MEM;
#pragma omp parallel for schedule(dynamic, 1)
  for (p = 0; p < np; ++p) {
    int le = pr_e[p];
    int t = token_list[pr_t[p] / k];
    oracle_expert_ffn(H, I, hidden + (int64_t)t * H,
                      hidden_scale + (int64_t)t * HB, w13[le], w13_scale[le],
                      w2[le], w2_scale[le], ys + (int64_t)p * H, NULL, NULL,
                      NULL);
  }

  /* (4) weighted scatter back to the tokens (pairs are in slot order) */
  acc = (double *)malloc(sizeof(double) * H);
  p = 0;
  for (r = 0; r < n_tokens; ++r) {
    for (n = 0; n < H; ++n) acc[n] = 0.0;
    while (p < np && pr_t[p] / k == r) {
      double wj = (double)w[pr_t[p]];
      for (n = 0; n < H; ++n) acc[n] += wj * ys[(int64_t)p * H + n];
      ++p;
    }
    for (n = 0; n < H; ++n)
      out[(int64_t)r * H + n] = oracle_bf16_from_double(acc[n]);
  }
  if (ids_out) memcpy(ids_out, ids, sizeof(int32_t) * (size_t)n_tokens * k);
  if (w_out) memcpy(w_out, w, sizeof(float) * (size_t)n_tokens * k);
  free(acc);
  free(ys);
  free(ids);
  free(w);
  free(pr_t);
  free(pr_e);
  return ORACLE_OK;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the parallel loops above (n < 1: leave unchanged).  Used to
 * time the oracle on one core. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ======================================================================== */
/* DSA TopK Indexer (paper Section 3.1.3): for each batch element b, score   */
/* every cached token j < seq_len[b] of the sequence against the query's    */
/* 64 heads and return the TopK highest-scoring tokens.                     */
/*   score(j) = sum over heads h of ReLU(q_h . k_j) * w_h                    */
/* Layouts: q [B, NH, D] e4m3; weights [B, NH] fp32; the key cache is paged: */
/* kc [num_pages, PS, D] e4m3 with per-token fp32 scales ks [num_pages, PS]; */
/* token j of sequence b is slot j % PS of page block_table[b][j / PS].     */
/* The scores decide which indices are returned, so they follow one fixed    */
/* fp32 sequence (the paper's kernel also keeps a scalar fp32 dot product    */
/* for bit-exactness):                                                        */
/*   kd[d]   = dec(kc[page, slot, d]) * ks[page, slot]      (one rounding)   */
/*   dot_h   = fused multiply-add chain over d ascending from 0 of          */
/*             dec(q[b, h, d]) * kd[d]                                        */
/*   score   = fused multiply-add chain over h ascending from 0 of          */
/*             max(dot_h, 0) * w[b, h]                                        */
/* Selection: the TopK tokens by score, larger first, equal scores to the    */
/* lower position; returned in ascending position order as physical cache   */
/* indices page * PS + slot, the rest of the TopK row padded with -1 (a      */
/* sequence of at most TopK tokens returns all of them).                     */
/* ======================================================================== */
typedef struct {
  int32_t B, NH, D, PS, topk, max_pages;
} oracle_dsa_shape;

int oracle_dsa_scores(const oracle_dsa_shape *s, const uint8_t *q, const float *w,
                      const uint8_t *kc, const float *ks, const int32_t *block_table,
                      const int32_t *seq_lens, int32_t b, float *scores) {
  int32_t L, j;
  if (!s || s->NH <= 0 || s->D <= 0 || s->D > 1024 || s->PS <= 0 || b < 0 || b >= s->B)
    return ORACLE_BAD_ARG;
  L = seq_lens[b];
  if (L < 0 || L > s->max_pages * s->PS) return ORACLE_BAD_ARG;
  {
    /* the query's codes decoded once (exact in fp32) */
    float *qd = (float *)malloc(sizeof(float) * (size_t)s->NH * s->D);
    int i;
    if (!qd) return ORACLE_NO_MEM;
    for (i = 0; i < s->NH * s->D; ++i)
      qd[i] = (float)oracle_e4m3_decode(q[(int64_t)b * s->NH * s->D + i]);
#pragma omp parallel for schedule(static)
    for (j = 0; j < L; ++j) {
      int64_t page = block_table[(int64_t)b * s->max_pages + j / s->PS];
      int slot = j % s->PS, h, d;
      const uint8_t *krow = kc + (page * s->PS + slot) * s->D;
      float scale = ks[page * s->PS + slot];
      float kd[1024];
      float acc = 0.0f;
      for (d = 0; d < s->D; ++d) kd[d] = (float)oracle_e4m3_decode(krow[d]) * scale;
      for (h = 0; h < s->NH; ++h) {
        const float *qh = qd + (int64_t)h * s->D;
        float dot = 0.0f, r;
        for (d = 0; d < s->D; ++d) dot = fmaf(qh[d], kd[d], dot);
        r = dot > 0.0f ? dot : 0.0f;
        acc = fmaf(r, w[(int64_t)b * s->NH + h], acc);
      }
      scores[j] = acc;
    }
    free(qd);
  }
  return ORACLE_OK;
}

typedef struct {
  float v;
  int32_t j;
} dsa_item;

static int dsa_by_score(const void *a, const void *b) {
  const dsa_item *x = (const dsa_item *)a, *y = (const dsa_item *)b;
  if (x->v > y->v) return -1;
  if (x->v < y->v) return 1;
  return x->j < y->j ? -1 : (x->j > y->j);
}

static int dsa_by_pos(const void *a, const void *b) {
  const dsa_item *x = (const dsa_item *)a, *y = (const dsa_item *)b;
  return x->j < y->j ? -1 : (x->j > y->j);
}

int oracle_dsa_topk(const oracle_dsa_shape *s, const uint8_t *q, const float *w,
                    const uint8_t *kc, const float *ks, const int32_t *block_table,
                    const int32_t *seq_lens, int32_t *out) {
  int32_t b;
  if (!s || s->B < 0 || s->topk <= 0) return ORACLE_BAD_ARG;
  for (b = 0; b < s->B; ++b) {
    int32_t L = seq_lens[b], n, i, rc;
    float *sc;
    dsa_item *it;
    int32_t *o = out + (int64_t)b * s->topk;
    if (L < 0 || L > s->max_pages * s->PS) return ORACLE_BAD_ARG;
    sc = (float *)malloc(sizeof(float) * (L > 0 ? L : 1));
    it = (dsa_item *)malloc(sizeof(dsa_item) * (L > 0 ? L : 1));
    if (!sc || !it) return ORACLE_NO_MEM;
    rc = oracle_dsa_scores(s, q, w, kc, ks, block_table, seq_lens, b, sc);
    if (rc) return rc;
    for (i = 0; i < L; ++i) {
      it[i].v = sc[i];
      it[i].j = i;
    }
    qsort(it, L, sizeof(dsa_item), dsa_by_score);
    n = L < s->topk ? L : s->topk;
    qsort(it, n, sizeof(dsa_item), dsa_by_pos);
    for (i = 0; i < s->topk; ++i) {
      if (i < n) {
        int32_t j = it[i].j;
        o[i] = block_table[(int64_t)b * s->max_pages + j / s->PS] * s->PS + j % s->PS;
      } else {
        o[i] = -1;
      }
    }
    free(sc);
    free(it);
  }
  return ORACLE_OK;
}
