/*
 * cold_oracle.c -- CPU checker for the COLD pre-ranking scoring path.
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the tests, the smoke
 * check and the bench's CPU-baseline leg load this library.  It shares no
 * code, header or table with the HIP library.
 *
 * It computes, plainly and in double precision, the forward pass that the
 * paper (Wang et al., "COLD: Towards the Next Generation of Pre-Ranking
 * System", DLP-KDD 2020) describes for scoring one candidate ad of one
 * request, one row at a time, with no blocking, fusion or reuse between rows:
 *
 *   1. id -> table row (direct ids, or hashed raw ids; the paper is silent on
 *      hashing, see orc_hash_row)
 *   2. embeddings of each feature group, concatenated in group order
 *      user, user behaviour sequence, ad, cross (GwEN input, Section 3.1);
 *      sequence groups are sum-pooled (Section 3.3, low precision)
 *   3. SE block importance weights, one scalar per group (Section 3.2, Eq. 2,
 *      read as squeeze -> FC -> ReLU -> FC -> sigmoid)
 *   4. optional top-k feature-group selection by importance (Section 3.2,
 *      feature group selection), per request
 *   5. field-wise reweighting v_i = s_i * e_i (Section 3.2)
 *   6. optional linear_log normalisation of the network input (Section 3.3,
 *      Eq. 3)
 *   7. fully connected network D_in x ... x n_out with ReLU hidden layers
 *      (Section 4.1) and a sigmoid (one output) or softmax (two outputs,
 *      CTR = probability of class 1) head.
 *
 * Stored parameters (fp32, bf16 or fp16 bit patterns) are converted exactly
 * to double; every arithmetic step is double.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F16 = 2 };
enum {
  ORC_OK = 0,
  ORC_BAD_ARG = -1,
  ORC_ID_RANGE = -2,
  ORC_NO_MEM = -3
};

typedef struct {
  int64_t n_requests;             /* Q */
  int64_t n_rows;                 /* R */
  int32_t n_user, n_seq, n_ad, n_cross;
  int32_t emb_dim;                /* d */
  int32_t se_hidden;              /* H */
  int32_t dtype;                  /* storage of tables and MLP weights */
  int32_t hashed;                 /* 0: int32 row ids; 1: uint64 raw ids */
  int32_t linear_log;             /* 0/1 */
  int32_t topk_k;                 /* 0: no group selection */
  int32_t n_layers;               /* number of fully connected layers */
  const int32_t *widths;          /* [n_layers + 1]; widths[0] = M*d */
  const int64_t *table_rows;      /* [M] */
  const void *const *tables;      /* [M] -> [rows][d] stored dtype */
  const float *se_w1;             /* [H][M] */
  const float *se_b1;             /* [H] */
  const float *se_w2;             /* [M][H] */
  const float *se_b2;             /* [M] */
  const void *const *mlp_w;       /* [n_layers] -> [out][in] stored dtype */
  const float *const *mlp_b;      /* [n_layers] -> [out] */
  const int32_t *req_off;         /* [Q + 1] */
  const void *user_ids;           /* [n_user][Q] */
  const void *ad_ids;             /* [n_ad][R] */
  const void *cross_ids;          /* [n_cross][R] */
  const int32_t *seq_off;         /* [n_seq * Q + 1], entry f*Q + q */
  const void *seq_ids;            /* [n_seq_ids] */
  int64_t n_seq_ids;
  const int32_t *cross_pairs;     /* [n_cross][2] (user field, ad field), or NULL:
                                     cross ids are then read from cross_ids */
  int32_t se_form;                /* 0: squeeze -> FC -> ReLU -> FC -> sigmoid;
                                     1: one FC over the concatenated embeddings,
                                        se_w1 [M][M*d], se_b1 [M] (Eq. 2 as printed) */
} orc_problem;

/* ---------------------------------------------------------------- dtypes */
static double from_f32(const void *p, int64_t i) { return (double)((const float *)p)[i]; }

static double from_bf16(const void *p, int64_t i) {
  /* bf16 is the upper half of an IEEE binary32 pattern */
  uint32_t bits = (uint32_t)((const uint16_t *)p)[i] << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

static double from_f16(const void *p, int64_t i) {
  /* IEEE binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits */
  uint16_t b = ((const uint16_t *)p)[i];
  int sign = b >> 15, ex = (b >> 10) & 31, fr = b & 1023;
  double v;
  if (ex == 0)
    v = ldexp((double)fr, -24);                 /* subnormal: fr * 2^-24 */
  else if (ex == 31)
    v = fr ? NAN : INFINITY;
  else
    v = ldexp((double)(1024 + fr), ex - 25);    /* (1 + fr/1024) * 2^(ex-15) */
  return sign ? -v : v;
}

static double load_stored(int dtype, const void *p, int64_t i) {
  if (dtype == ORC_BF16) return from_bf16(p, i);
  if (dtype == ORC_F16) return from_f16(p, i);
  return from_f32(p, i);
}

/* The decoder above on n stored values (for the tests that pin it against
 * an independent widening of every 16-bit pattern). */
int orc_decode_stored(int32_t dtype, const void *p, int64_t n, double *out) {
  if ((dtype != ORC_F32 && dtype != ORC_BF16 && dtype != ORC_F16) || n < 0 || (n > 0 && (!p || !out)))
    return ORC_BAD_ARG;
  for (int64_t i = 0; i < n; ++i) out[i] = load_stored(dtype, p, i);
  return ORC_OK;
}

/* --------------------------------------------------------- id resolution */
/* SplitMix64 output function (Steele, Lea, Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014). */
uint64_t orc_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

/* Hashed tables: a raw 64-bit id of feature group g lands in row
 * mix64(raw XOR salt_g) mod rows, with salt_g = (g + 1) * 0x9e3779b97f4a7c15
 * (mod 2^64), the SplitMix64 increment.  The paper does not describe id
 * hashing; this is the reading used throughout. */
uint64_t orc_hash_row(uint64_t raw, int32_t g, uint64_t rows) {
  uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ULL;
  return orc_mix64(raw ^ salt) % rows;
}

/* A user x ad cross feature formed from the raw ids of one user field and
 * one ad field (the paper forms its cross features on the CPU and does not
 * say how; this is the reading used throughout): the pair's 64-bit key is
 * mix64(user id) XOR ad id, with 32-bit ids taken as unsigned, and the key
 * is hashed into the cross group's table like a raw id (orc_hash_row). */
uint64_t orc_cross_key(uint64_t user_id, uint64_t ad_id) {
  return orc_mix64(user_id) ^ ad_id;
}

static uint64_t raw_id(const orc_problem *p, const void *ids, int64_t i) {
  if (p->hashed) return ((const uint64_t *)ids)[i];
  return (uint64_t)(uint32_t)((const int32_t *)ids)[i];
}

/* row of group g for an id stored at element i of column array `ids`;
 * returns -1 for a direct id outside [0, rows) */
static int64_t resolve(const orc_problem *p, const void *ids, int64_t i, int32_t g) {
  uint64_t rows = (uint64_t)p->table_rows[g];
  if (p->hashed) return (int64_t)orc_hash_row(((const uint64_t *)ids)[i], g, rows);
  int32_t id = ((const int32_t *)ids)[i];
  if (id < 0 || (uint64_t)id >= rows) return -1;
  return id;
}

/* ------------------------------------------------------------ operators */
/* Eq. 3: -log(-x) - 1 for x < -1; x on [-1, 1]; log(x) + 1 for x > 1
 * (natural log: the only base for which the pieces join with slope 1). */
double orc_linear_log(double x) {
  if (x < -1.0) return -log(-x) - 1.0;
  if (x > 1.0) return log(x) + 1.0;
  return x;
}

static double sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }

/* request that row r belongs to (last q with req_off[q] <= r < req_off[q+1]) */
static int64_t request_of(const orc_problem *p, int64_t r) {
  for (int64_t q = 0; q < p->n_requests; ++q)
    if (p->req_off[q] <= r && r < p->req_off[q + 1]) return q;
  return -1;
}

/* Embeddings of all M groups of row r (request q) into e[M*d]; the resolved
 * table row of each single-valued group into rows_out[M] (-1 for sequence
 * groups).  Returns ORC_OK or ORC_ID_RANGE. */
static int row_embeddings(const orc_problem *p, int64_t r, int64_t q, double *e,
                          int64_t *rows_out) {
  const int d = p->emb_dim;
  const int64_t Q = p->n_requests, R = p->n_rows;
  int32_t g = 0;
  for (int32_t f = 0; f < p->n_user; ++f, ++g) {
    int64_t row = resolve(p, p->user_ids, (int64_t)f * Q + q, g);
    if (row < 0) return ORC_ID_RANGE;
    rows_out[g] = row;
    for (int k = 0; k < d; ++k)
      e[g * d + k] = load_stored(p->dtype, p->tables[g], row * d + k);
  }
  for (int32_t f = 0; f < p->n_seq; ++f, ++g) {
    int64_t lo = p->seq_off[(int64_t)f * Q + q], hi = p->seq_off[(int64_t)f * Q + q + 1];
    rows_out[g] = -1;
    for (int k = 0; k < d; ++k) e[g * d + k] = 0.0;
    for (int64_t j = lo; j < hi; ++j) {  /* sum-pooling, in sequence order */
      int64_t row = resolve(p, p->seq_ids, j, g);
      if (row < 0) return ORC_ID_RANGE;
      for (int k = 0; k < d; ++k)
        e[g * d + k] += load_stored(p->dtype, p->tables[g], row * d + k);
    }
  }
  for (int32_t f = 0; f < p->n_ad; ++f, ++g) {
    int64_t row = resolve(p, p->ad_ids, (int64_t)f * R + r, g);
    if (row < 0) return ORC_ID_RANGE;
    rows_out[g] = row;
    for (int k = 0; k < d; ++k)
      e[g * d + k] = load_stored(p->dtype, p->tables[g], row * d + k);
  }
  for (int32_t f = 0; f < p->n_cross; ++f, ++g) {
    int64_t row;
    if (p->cross_pairs) {
      uint64_t key = orc_cross_key(raw_id(p, p->user_ids, (int64_t)p->cross_pairs[2 * f] * Q + q),
                                   raw_id(p, p->ad_ids, (int64_t)p->cross_pairs[2 * f + 1] * R + r));
      row = (int64_t)orc_hash_row(key, g, (uint64_t)p->table_rows[g]);
    } else {
      row = resolve(p, p->cross_ids, (int64_t)f * R + r, g);
    }
    if (row < 0) return ORC_ID_RANGE;
    rows_out[g] = row;
    for (int k = 0; k < d; ++k)
      e[g * d + k] = load_stored(p->dtype, p->tables[g], row * d + k);
  }
  return ORC_OK;
}

/* SE block (Eq. 2, Hu et al. form): z_g = mean_k e_g[k];
 * h = ReLU(W1 z + b1); s = sigmoid(W2 h + b2). */
static void se_weights(const orc_problem *p, const double *e, double *z, double *h,
                       double *s) {
  const int d = p->emb_dim, H = p->se_hidden;
  const int M = p->n_user + p->n_seq + p->n_ad + p->n_cross;
  if (p->se_form == 1) {
    /* Eq. 2 as printed: s = sigmoid(W [e_1, ..., e_M] + b), one fully
     * connected layer from the whole concatenated embedding to M weights */
    const int64_t D = (int64_t)M * d;
    for (int g = 0; g < M; ++g) {
      double acc = (double)p->se_b1[g];
      for (int64_t j = 0; j < D; ++j) acc += (double)p->se_w1[(int64_t)g * D + j] * e[j];
      s[g] = sigmoid(acc);
    }
    return;
  }
  for (int g = 0; g < M; ++g) {
    double acc = 0.0;
    for (int k = 0; k < d; ++k) acc += e[g * d + k];
    z[g] = acc / d;
  }
  for (int j = 0; j < H; ++j) {
    double acc = (double)p->se_b1[j];
    for (int g = 0; g < M; ++g) acc += (double)p->se_w1[(int64_t)j * M + g] * z[g];
    h[j] = acc > 0.0 ? acc : 0.0;
  }
  for (int g = 0; g < M; ++g) {
    double acc = (double)p->se_b2[g];
    for (int j = 0; j < H; ++j) acc += (double)p->se_w2[(int64_t)g * H + j] * h[j];
    s[g] = sigmoid(acc);
  }
}

/* Fully connected network on x[widths[0]]; returns CTR. */
static double mlp_ctr(const orc_problem *p, const double *x, double *buf_a, double *buf_b) {
  int L = p->n_layers;
  const double *in = x;
  double *out = buf_a;
  for (int l = 0; l < L; ++l) {
    int fi = p->widths[l], fo = p->widths[l + 1];
    for (int o = 0; o < fo; ++o) {
      double acc = (double)p->mlp_b[l][o];
      for (int i = 0; i < fi; ++i)
        acc += load_stored(p->dtype, p->mlp_w[l], (int64_t)o * fi + i) * in[i];
      out[o] = (l < L - 1 && acc < 0.0) ? 0.0 : acc;   /* ReLU on hidden layers */
    }
    in = out;
    out = (out == buf_a) ? buf_b : buf_a;
  }
  int n_out = p->widths[L];
  if (n_out == 1) return sigmoid(in[0]);
  /* softmax over the outputs, probability of class 1 */
  double mx = in[0];
  for (int o = 1; o < n_out; ++o) mx = in[o] > mx ? in[o] : mx;
  double den = 0.0;
  for (int o = 0; o < n_out; ++o) den += exp(in[o] - mx);
  return exp(in[1] - mx) / den;
}

static int check_problem(const orc_problem *p) {
  if (!p || p->n_requests < 0 || p->n_rows < 0 || p->emb_dim <= 0 || p->se_hidden <= 0)
    return ORC_BAD_ARG;
  int M = p->n_user + p->n_seq + p->n_ad + p->n_cross;
  if (M <= 0 || p->n_layers <= 0 || p->widths[0] != M * p->emb_dim) return ORC_BAD_ARG;
  int n_out = p->widths[p->n_layers];
  if (n_out != 1 && n_out != 2) return ORC_BAD_ARG;
  if (p->topk_k < 0) return ORC_BAD_ARG;
  if (p->req_off[0] != 0 || p->req_off[p->n_requests] != p->n_rows) return ORC_BAD_ARG;
  for (int64_t q = 0; q < p->n_requests; ++q)
    if (p->req_off[q + 1] < p->req_off[q]) return ORC_BAD_ARG;
  if (p->n_seq > 0) {
    int64_t n = (int64_t)p->n_seq * p->n_requests;
    if (p->seq_off[0] != 0 || p->seq_off[n] != p->n_seq_ids) return ORC_BAD_ARG;
    for (int64_t i = 0; i < n; ++i)
      if (p->seq_off[i + 1] < p->seq_off[i]) return ORC_BAD_ARG;
  }
  return ORC_OK;
}

/* Per-request group mask (Section 3.2, feature group selection): importance
 * I_g = mean over the request's rows of s_g; keep the k groups with the
 * largest I_g, ties to the lower group index.  imp[Q][M], mask[Q][M]. */
static int group_masks(const orc_problem *p, double *imp, uint8_t *mask, int n_threads) {
  const int M = p->n_user + p->n_seq + p->n_ad + p->n_cross;
  const int d = p->emb_dim, H = p->se_hidden;
  const int64_t Q = p->n_requests;
  int status = ORC_OK;
  for (int64_t q = 0; q < Q; ++q) {
    int64_t lo = p->req_off[q], hi = p->req_off[q + 1];
    double *sums = calloc((size_t)M, sizeof(double));
    double *srow = malloc(sizeof(double) * (size_t)(hi > lo ? hi - lo : 1) * M);
    if (!sums || !srow) { free(sums); free(srow); return ORC_NO_MEM; }
#pragma omp parallel for schedule(static) num_threads(n_threads)
    for (int64_t r = lo; r < hi; ++r) {
      double *e = malloc(sizeof(double) * (size_t)M * d);
      double *z = malloc(sizeof(double) * M), *h = malloc(sizeof(double) * H);
      int64_t *rows = malloc(sizeof(int64_t) * M);
      if (row_embeddings(p, r, q, e, rows) != ORC_OK) {
#pragma omp critical
        status = ORC_ID_RANGE;
      } else {
        se_weights(p, e, z, h, srow + (r - lo) * M);
      }
      free(e); free(z); free(h); free(rows);
    }
    if (status != ORC_OK) { free(sums); free(srow); return status; }
    for (int64_t r = lo; r < hi; ++r)           /* sum in row order */
      for (int g = 0; g < M; ++g) sums[g] += srow[(r - lo) * M + g];
    for (int g = 0; g < M; ++g) imp[q * M + g] = hi > lo ? sums[g] / (double)(hi - lo) : 0.0;
    for (int g = 0; g < M; ++g) {
      /* rank of g in the order (importance descending, index ascending) */
      int rank = 0;
      for (int o = 0; o < M; ++o) {
        double io = imp[q * M + o], ig = imp[q * M + g];
        if (io > ig || (io == ig && o < g)) ++rank;
      }
      mask[q * M + g] = rank < p->topk_k ? 1 : 0;
    }
    free(sums); free(srow);
  }
  return ORC_OK;
}

/*
 * Score the rows listed in sample[n_sample].
 *   scores[n_sample]                CTR
 *   rows_out[n_sample][M]   (opt.)  resolved table row per group (-1: sequence)
 *   s_out[n_sample][M]      (opt.)  SE importance weights (before any mask)
 *   x_out[n_sample][D_in]   (opt.)  network input (after reweighting, mask and
 *                                   linear_log)
 *   z_out[n_sample][M]      (opt.)  squeeze z of the SE block (zero for the
 *                                   one-layer form, which has none)
 *   imp_out[Q][M], mask_out[Q][M] (opt., only when topk_k > 0)
 * Returns ORC_OK, ORC_BAD_ARG, ORC_ID_RANGE or ORC_NO_MEM.
 */
int orc_score(const orc_problem *p, const int64_t *sample, int64_t n_sample, double *scores,
              int64_t *rows_out, double *s_out, double *x_out, double *z_out,
              double *imp_out, uint8_t *mask_out, int n_threads) {
  int st = check_problem(p);
  if (st != ORC_OK) return st;
  const int M = p->n_user + p->n_seq + p->n_ad + p->n_cross;
  const int d = p->emb_dim, H = p->se_hidden, D = M * d;
  const int64_t Q = p->n_requests;
  if (n_threads < 1) n_threads = 1;
  for (int64_t i = 0; i < n_sample; ++i)
    if (sample[i] < 0 || sample[i] >= p->n_rows) return ORC_BAD_ARG;

  double *imp = NULL;
  uint8_t *mask = NULL;
  if (p->topk_k > 0) {
    imp = malloc(sizeof(double) * (size_t)(Q > 0 ? Q : 1) * M);
    mask = malloc((size_t)(Q > 0 ? Q : 1) * M);
    if (!imp || !mask) { free(imp); free(mask); return ORC_NO_MEM; }
    st = group_masks(p, imp, mask, n_threads);
    if (st != ORC_OK) { free(imp); free(mask); return st; }
    if (imp_out) memcpy(imp_out, imp, sizeof(double) * (size_t)Q * M);
    if (mask_out) memcpy(mask_out, mask, (size_t)Q * M);
  }
  int maxw = 0;
  for (int l = 0; l <= p->n_layers; ++l) maxw = p->widths[l] > maxw ? p->widths[l] : maxw;

  int status = ORC_OK;
#pragma omp parallel for schedule(static) num_threads(n_threads)
  for (int64_t i = 0; i < n_sample; ++i) {
    int64_t r = sample[i];
    int64_t q = request_of(p, r);
    double *e = malloc(sizeof(double) * (size_t)D);
    double *x = malloc(sizeof(double) * (size_t)D);
    double *z = malloc(sizeof(double) * M), *h = malloc(sizeof(double) * H);
    double *s = malloc(sizeof(double) * M);
    double *ba = malloc(sizeof(double) * maxw), *bb = malloc(sizeof(double) * maxw);
    int64_t *rows = malloc(sizeof(int64_t) * M);
    if (row_embeddings(p, r, q, e, rows) != ORC_OK) {
#pragma omp critical
      status = ORC_ID_RANGE;
    } else {
      se_weights(p, e, z, h, s);
      for (int g = 0; g < M; ++g) {
        double keep = mask ? (double)mask[q * M + g] : 1.0;
        for (int k = 0; k < d; ++k) {
          double v = s[g] * keep * e[g * d + k];        /* v_i = s_i e_i */
          x[g * d + k] = p->linear_log ? orc_linear_log(v) : v;
        }
      }
      scores[i] = mlp_ctr(p, x, ba, bb);
      if (rows_out) memcpy(rows_out + i * M, rows, sizeof(int64_t) * M);
      if (s_out) memcpy(s_out + i * M, s, sizeof(double) * M);
      if (x_out) memcpy(x_out + i * D, x, sizeof(double) * D);
      if (z_out) {
        if (p->se_form == 1) memset(z_out + i * M, 0, sizeof(double) * M);
        else memcpy(z_out + i * M, z, sizeof(double) * M);
      }
    }
    free(e); free(x); free(z); free(h); free(s); free(ba); free(bb); free(rows);
  }
  free(imp);
  free(mask);
  return status;
}
