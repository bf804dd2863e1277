/*
 * kvo.c -- CPU oracle for the KV rebuild.  TEST INFRASTRUCTURE ONLY: the
 * product library never links or calls this file; tests, the smoke check and
 * the benchmark's CPU baseline do.
 *
 * Plain definition of the rebuild (Sec. 4.2 Handover step 5 and Sec. 4.3 LLM
 * Context Recovery: rebuild request KV from logged token prefixes into the
 * retained raw arena; Sec. 2.3 Finding 2: complete KV is never reused, so every
 * listed slot is recomputed and overwritten).  The model forward the paper
 * leaves unstated is a Llama-style pre-norm decoder:
 *
 *   x_p = E[t_p]                                        (fp32 residual stream)
 *   per layer:
 *     a_p  = rnd(g_attn * x_p / sqrt(mean(x_p^2) + eps))
 *     q, k, v = Wq a_p, Wk a_p, Wv a_p
 *     RoPE (NeoX half-split, pairs (i, i+d/2), angle p * theta^(-2i/d) in fp64,
 *           cos/sin rounded to fp32) on q and k
 *     K^_p = rnd(k_rot), V^_p = rnd(v)  -> arena slot (table[p / B], p % B)
 *     Q^_p = rnd(q_rot)
 *     attention per q head h over kv head h / (nq / nkv), positions j <= p,
 *       reading K^/V^ back from the arena:  o = sum_j softmax_j(Q^.K^_j/sqrt d) V^_j
 *     u_p = rnd(o);  x_p += Wo u_p
 *     b_p = rnd(g_ffn * x_p / sqrt(mean(x_p^2) + eps))
 *     h_p = rnd(silu(Wg b_p) * (Wu b_p));  x_p += Wd h_p
 *
 * Every reduction is a plain sequential fp64 sum; every op output is rounded
 * to fp32 before the next op; rnd() is the identity for fp32 models and
 * fp32 -> bf16 round-to-nearest-even for bf16 models.  KVO_F64 rounds nothing.
 *
 * Optional mode round_p: the attention weights are rounded like an op output
 * before both the weighted sum of V^ and the denominator.  Softmax is
 * unchanged by scaling every weight of a row by one factor, and rounding to
 * fp32 or bf16 commutes with scaling by a power of two, so the weights are
 * taken relative to a power of two of the row maximum: with c = ceil(max_j
 * z_j log2 e), w_j = rnd(fp32(2^(z_j log2 e - c))).  The result then does not
 * depend on which power of two anchors the row (any integer c gives the same
 * rounded weights up to that factor), which is what lets an online softmax
 * that raises its anchor tile by tile round exactly these weights.  It models
 * a freedom the GPU path declares (its P.V product takes P in the model
 * dtype); the definition above is the mode off.
 */
#include "kvo.h"

#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ */
/* scalar conversions                                                  */
/* ------------------------------------------------------------------ */
static double bf16_bits_to_double(uint16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

uint16_t kvo_round_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u); /* NaN stays NaN */
  u += 0x7fffu + ((u >> 16) & 1u); /* round half to even on the dropped 16 bits */
  return (uint16_t)(u >> 16);
}

int kvo_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* op output -> working precision (fp32), except in the fp64 pin mode */
static double to_work(double v, int dt) { return dt == KVO_F64 ? v : (double)(float)v; }

/* the declared rounding sites: working precision, then the model dtype */
static double rnd(double v, int dt) {
  if (dt == KVO_F64) return v;
  float f = (float)v;
  if (dt == KVO_BF16) return bf16_bits_to_double(kvo_round_bf16(f));
  return (double)f;
}

static double load(const void* p, int dt, int64_t i) {
  if (dt == KVO_BF16) return bf16_bits_to_double(((const uint16_t*)p)[i]);
  if (dt == KVO_F32) return (double)((const float*)p)[i];
  return ((const double*)p)[i];
}

/* v must already be representable in dt (it went through rnd) */
static void store(void* p, int dt, int64_t i, double v) {
  if (dt == KVO_BF16)
    ((uint16_t*)p)[i] = kvo_round_bf16((float)v);
  else if (dt == KVO_F32)
    ((float*)p)[i] = (float)v;
  else
    ((double*)p)[i] = v;
}

/* sum_k W[row][k] * a[k], plain order */
static double dot_row(const void* w, int dt, int64_t row, int64_t K, const double* a) {
  double s = 0.0;
  int64_t k;
  if (dt == KVO_BF16) {
    const uint16_t* p = (const uint16_t*)w + row * K;
    for (k = 0; k < K; ++k) s += bf16_bits_to_double(p[k]) * a[k];
  } else if (dt == KVO_F32) {
    const float* p = (const float*)w + row * K;
    for (k = 0; k < K; ++k) s += (double)p[k] * a[k];
  } else {
    const double* p = (const double*)w + row * K;
    for (k = 0; k < K; ++k) s += p[k] * a[k];
  }
  return s;
}

/* ------------------------------------------------------------------ */
/* per-op building blocks (each works on `cnt` rows)                   */
/* ------------------------------------------------------------------ */

/* out[r][i] = to_work(W[i] . A[r]) for W [N, K] */
static void project(const void* W, int dt, int64_t N, int64_t K, const double* A,
                    int64_t cnt, double* out) {
  int64_t idx;
#pragma omp parallel for schedule(static)
  for (idx = 0; idx < cnt * N; ++idx) {
    int64_t r = idx / N, i = idx % N;
    out[idx] = to_work(dot_row(W, dt, i, K, A + r * K), dt);
  }
}

/* out[r][i] = to_work(W[i] . A[r] + b[i]): the bias joins the sum before the
 * single rounding */
static void project_bias(const void* W, const void* b, int dt, int64_t N, int64_t K,
                         const double* A, int64_t cnt, double* out) {
  int64_t idx;
#pragma omp parallel for schedule(static)
  for (idx = 0; idx < cnt * N; ++idx) {
    int64_t r = idx / N, i = idx % N;
    out[idx] = to_work(dot_row(W, dt, i, K, A + r * K) + load(b, dt, i), dt);
  }
}

/* per-head RMSNorm with a gain over the head dims, in place on [cnt][nh][d];
 * the result stays in working precision (RoPE and the rounding follow) */
static void head_rmsnorm(double* u, const void* g, int dt, int64_t cnt, int64_t nh, int64_t d,
                         double eps) {
  int64_t idx;
#pragma omp parallel for schedule(static)
  for (idx = 0; idx < cnt * nh; ++idx) {
    double* hu = u + idx * d;
    double ss = 0.0, inv;
    int64_t e;
    for (e = 0; e < d; ++e) ss += hu[e] * hu[e];
    inv = 1.0 / sqrt(ss / (double)d + eps);
    for (e = 0; e < d; ++e) hu[e] = to_work(load(g, dt, e) * hu[e] * inv, dt);
  }
}

/* RMSNorm with gain, one rounding at the end */
static void rmsnorm(const double* x, const void* g, int dt, int64_t H, double eps,
                    int64_t cnt, double* out) {
  int64_t r;
#pragma omp parallel for schedule(static)
  for (r = 0; r < cnt; ++r) {
    const double* xr = x + r * H;
    double ss = 0.0, inv;
    int64_t j;
    for (j = 0; j < H; ++j) ss += xr[j] * xr[j];
    inv = 1.0 / sqrt(ss / (double)H + eps);
    for (j = 0; j < H; ++j) out[r * H + j] = rnd(load(g, dt, j) * xr[j] * inv, dt);
  }
}

/* NeoX half-split rotary embedding of every head of one row at position pos */
static void rope_row(double* u, int nheads, int d, int64_t pos, double theta, int dt) {
  int h, i, half = d / 2;
  for (i = 0; i < half; ++i) {
    double inv_freq = pow(theta, -(double)(2 * i) / (double)d);
    double phi = (double)pos * inv_freq;
    double c = cos(phi), s = sin(phi);
    if (dt != KVO_F64) { c = (double)(float)c; s = (double)(float)s; }
    for (h = 0; h < nheads; ++h) {
      double* hu = u + (int64_t)h * d;
      double a = hu[i], b = hu[i + half];
      hu[i] = to_work(a * c - b * s, dt);
      hu[i + half] = to_work(b * c + a * s, dt);
    }
  }
}

static int64_t arena_off(const kvo_model* m, const kvo_arena* ar, int l, int kv, int64_t slot) {
  return ((((int64_t)l * 2 + kv) * ar->num_blocks * ar->block_size + slot) * m->num_kv_heads) *
         m->head_dim;
}

static int64_t slot_of(const kvo_arena* ar, const int32_t* table, int64_t p) {
  return (int64_t)table[p / ar->block_size] * ar->block_size + p % ar->block_size;
}

/* ------------------------------------------------------------------ */
/* one layer over positions [p0, p0 + cnt) of one request              */
/* ------------------------------------------------------------------ */
static void layer_step(const kvo_model* m, const kvo_layer* lw, int l, double* x, int64_t p0,
                       int64_t cnt, const int32_t* table, kvo_arena* ar, int kv_only,
                       double* scratch) {
  const int dt = m->dtype;
  const int64_t H = m->hidden, d = m->head_dim, nq = m->num_q_heads, nkv = m->num_kv_heads;
  const int64_t F = m->ffn_dim, g = nq / nkv;
  double *a = scratch, *q = a + cnt * H, *k = q + cnt * nq * d, *v = k + cnt * nkv * d;
  double *u = v + cnt * nkv * d, *gate = u + cnt * nq * d, *up = gate + cnt * F;
  int64_t r, idx;

  /* attention RMSNorm and Q/K/V projections */
  rmsnorm(x, lw->attn_norm, dt, H, m->rms_eps, cnt, a);
  if (m->qkv_bias) {
    project_bias(lw->wq, lw->bq, dt, nq * d, H, a, cnt, q);
    project_bias(lw->wk, lw->bk, dt, nkv * d, H, a, cnt, k);
    project_bias(lw->wv, lw->bv, dt, nkv * d, H, a, cnt, v);
  } else {
    project(lw->wq, dt, nq * d, H, a, cnt, q);
    project(lw->wk, dt, nkv * d, H, a, cnt, k);
    project(lw->wv, dt, nkv * d, H, a, cnt, v);
  }
  if (m->qk_norm) {
    head_rmsnorm(q, lw->q_norm, dt, cnt, nq, d, m->rms_eps);
    head_rmsnorm(k, lw->k_norm, dt, cnt, nkv, d, m->rms_eps);
  }

  /* RoPE on q and k, round, write K^ / V^ to the arena */
#pragma omp parallel for schedule(static)
  for (r = 0; r < cnt; ++r) {
    const int64_t p = p0 + r;
    const int64_t slot = slot_of(ar, table, p);
    int64_t e;
    rope_row(q + r * nq * d, (int)nq, (int)d, p, m->rope_theta, dt);
    rope_row(k + r * nkv * d, (int)nkv, (int)d, p, m->rope_theta, dt);
    for (e = 0; e < nq * d; ++e) q[r * nq * d + e] = rnd(q[r * nq * d + e], dt);
    for (e = 0; e < nkv * d; ++e) {
      store(ar->base, dt, arena_off(m, ar, l, 0, slot) + e, rnd(k[r * nkv * d + e], dt));
      store(ar->base, dt, arena_off(m, ar, l, 1, slot) + e, rnd(v[r * nkv * d + e], dt));
    }
  }
  if (kv_only) return;

  /* causal GQA attention, K^/V^ read back from the arena */
#pragma omp parallel for schedule(dynamic, 1)
  for (idx = 0; idx < cnt * nq; ++idx) {
    const int64_t r = idx / nq, h = idx % nq, kvh = h / g, p = p0 + r;
    const double* qh = q + r * nq * d + h * d;
    const double scale = 1.0 / sqrt((double)d);
    double* z = (double*)malloc(sizeof(double) * (size_t)(p + 1));
    double zmax = -INFINITY, den = 0.0;
    int64_t j, e;
    for (j = 0; j <= p; ++j) {
      const int64_t ko = arena_off(m, ar, l, 0, slot_of(ar, table, j)) + kvh * d;
      double s = 0.0;
      for (e = 0; e < d; ++e) s += qh[e] * load(ar->base, dt, ko + e);
      z[j] = s * scale;
      if (z[j] > zmax) zmax = z[j];
    }
    if (m->round_p) {
      const double c = ceil(zmax * M_LOG2E);
      for (j = 0; j <= p; ++j) {
        z[j] = rnd(to_work(exp2(z[j] * M_LOG2E - c), dt), dt);
        den += z[j];
      }
    } else {
      for (j = 0; j <= p; ++j) {
        z[j] = exp(z[j] - zmax);
        den += z[j];
      }
    }
    for (e = 0; e < d; ++e) {
      double o = 0.0;
      for (j = 0; j <= p; ++j) {
        const int64_t vo = arena_off(m, ar, l, 1, slot_of(ar, table, j)) + kvh * d;
        o += z[j] * load(ar->base, dt, vo + e);
      }
      u[r * nq * d + h * d + e] = rnd(to_work(o / den, dt), dt);
    }
    free(z);
  }

  /* output projection into the residual */
  project(lw->wo, dt, H, nq * d, u, cnt, a);
  for (idx = 0; idx < cnt * H; ++idx) x[idx] = to_work(x[idx] + a[idx], dt);

  /* FFN RMSNorm, SwiGLU, down projection into the residual */
  rmsnorm(x, lw->ffn_norm, dt, H, m->rms_eps, cnt, a);
  project(lw->w_gate, dt, F, H, a, cnt, gate);
  project(lw->w_up, dt, F, H, a, cnt, up);
  for (idx = 0; idx < cnt * F; ++idx) {
    const double gv = gate[idx];
    const double silu = gv / (1.0 + exp(-gv));
    gate[idx] = rnd(to_work(silu * up[idx], dt), dt);
  }
  project(lw->w_down, dt, H, F, gate, cnt, a);
  for (idx = 0; idx < cnt * H; ++idx) x[idx] = to_work(x[idx] + a[idx], dt);
}

static size_t scratch_elems(const kvo_model* m, int64_t cnt) {
  const int64_t H = m->hidden, d = m->head_dim;
  return (size_t)(cnt * (H + 2 * m->num_q_heads * d + 2 * m->num_kv_heads * d + 2 * m->ffn_dim));
}

static int check_args(const kvo_model* m, const int32_t* tokens, const int32_t* lens, int32_t R,
                      const int32_t* tables, int32_t max_blocks, const kvo_arena* ar) {
  int64_t off = 0;
  int32_t r;
  if (!m || R < 0 || !ar || !ar->base || ar->block_size <= 0) return -1;
  if (m->num_q_heads % m->num_kv_heads != 0 || m->head_dim % 2 != 0) return -1;
  for (r = 0; r < R; ++r) {
    int64_t n = lens[r], p, b;
    if (n < 0 || (n + ar->block_size - 1) / ar->block_size > max_blocks) return -1;
    for (p = 0; p < n; ++p)
      if (tokens[off + p] < 0 || tokens[off + p] >= m->vocab) return -1;
    for (b = 0; b < (n + ar->block_size - 1) / ar->block_size; ++b) {
      int32_t blk = tables[(int64_t)r * max_blocks + b];
      if (blk < 0 || blk >= ar->num_blocks) return -1;
    }
    off += n;
  }
  return 0;
}

static void embed_rows(const kvo_model* m, const void* embed, const int32_t* tok, int64_t cnt,
                       double* x) {
  const int64_t H = m->hidden;
  int64_t r, j;
  for (r = 0; r < cnt; ++r)
    for (j = 0; j < H; ++j) x[r * H + j] = to_work(load(embed, m->dtype, (int64_t)tok[r] * H + j), m->dtype);
}

int kvo_rebuild_from(const kvo_model* m, const void* embed, const kvo_layer* layers,
                     const int32_t* tokens, const int32_t* lens, const int32_t* starts,
                     int32_t num_requests, const int32_t* block_tables, int32_t max_blocks,
                     kvo_arena* arena, double* final_hidden) {
  int64_t off = 0;
  int32_t r;
  if (!m || !lens || !starts || num_requests < 0 || !arena || !arena->base || arena->block_size <= 0)
    return -1;
  if (m->num_q_heads % m->num_kv_heads != 0 || m->head_dim % 2 != 0) return -1;
  for (r = 0; r < num_requests; ++r) {
    const int64_t n = lens[r], s = starts[r];
    int64_t p, b;
    if (n < 0 || s < 0 || s > n || (n + arena->block_size - 1) / arena->block_size > max_blocks) return -1;
    for (p = 0; p < n - s; ++p)
      if (tokens[off + p] < 0 || tokens[off + p] >= m->vocab) return -1;
    for (b = 0; b < (n + arena->block_size - 1) / arena->block_size; ++b) {
      const int32_t blk = block_tables[(int64_t)r * max_blocks + b];
      if (blk < 0 || blk >= arena->num_blocks) return -1;
    }
    off += n - s;
  }
  off = 0;
  for (r = 0; r < num_requests; ++r) {
    const int64_t s = starts[r], cnt = lens[r] - starts[r], H = m->hidden;
    const int32_t* table = block_tables + (int64_t)r * max_blocks;
    double *x, *scratch;
    int l;
    if (cnt == 0) continue;
    x = (double*)malloc(sizeof(double) * (size_t)(cnt * H));
    scratch = (double*)malloc(sizeof(double) * scratch_elems(m, cnt));
    embed_rows(m, embed, tokens + off, cnt, x);
    for (l = 0; l < m->num_layers; ++l) {
      const int kv_only = (l == m->num_layers - 1) && final_hidden == NULL;
      layer_step(m, &layers[l], l, x, s, cnt, table, arena, kv_only, scratch);
    }
    if (final_hidden) memcpy(final_hidden + off * H, x, sizeof(double) * (size_t)(cnt * H));
    free(scratch);
    free(x);
    off += cnt;
  }
  return 0;
}

/* Progress lines on stderr, one per layer of every request of at least 256
 * tokens, when the environment sets KVO_PROGRESS=1 (long test runs report
 * that they are alive); nothing else depends on it. */
static int progress_on(void) {
  const char* e = getenv("KVO_PROGRESS");
  return e != NULL && e[0] == '1';
}

int kvo_rebuild(const kvo_model* m, const void* embed, const kvo_layer* layers,
                const int32_t* tokens, const int32_t* lens, int32_t num_requests,
                const int32_t* block_tables, int32_t max_blocks, kvo_arena* arena,
                double* final_hidden) {
  int64_t off = 0;
  int32_t r;
  const int progress = progress_on();
  if (check_args(m, tokens, lens, num_requests, block_tables, max_blocks, arena)) return -1;
  for (r = 0; r < num_requests; ++r) {
    const int64_t n = lens[r], H = m->hidden;
    const int32_t* table = block_tables + (int64_t)r * max_blocks;
    double *x, *scratch;
    int l;
    if (n == 0) continue;
    x = (double*)malloc(sizeof(double) * (size_t)(n * H));
    scratch = (double*)malloc(sizeof(double) * scratch_elems(m, n));
    embed_rows(m, embed, tokens + off, n, x);
    for (l = 0; l < m->num_layers; ++l) {
      const int kv_only = (l == m->num_layers - 1) && final_hidden == NULL;
      layer_step(m, &layers[l], l, x, 0, n, table, arena, kv_only, scratch);
      if (progress && n >= 256) {
        fprintf(stderr, "[oracle] request %d (%lld tokens): layer %d of %d\n", (int)r, (long long)n, l + 1,
                m->num_layers);
        fflush(stderr);
      }
    }
    if (final_hidden) memcpy(final_hidden + off * H, x, sizeof(double) * (size_t)(n * H));
    free(scratch);
    free(x);
    off += n;
  }
  return 0;
}

int kvo_decode(const kvo_model* m, const void* embed, const kvo_layer* layers,
               const int32_t* tokens, const int32_t* lens, int32_t num_requests,
               const int32_t* block_tables, int32_t max_blocks, kvo_arena* arena,
               double* final_hidden) {
  int64_t off = 0;
  int32_t r;
  if (check_args(m, tokens, lens, num_requests, block_tables, max_blocks, arena)) return -1;
  for (r = 0; r < num_requests; ++r) {
    const int64_t n = lens[r], H = m->hidden;
    const int32_t* table = block_tables + (int64_t)r * max_blocks;
    double* x = (double*)malloc(sizeof(double) * (size_t)H);
    double* scratch = (double*)malloc(sizeof(double) * scratch_elems(m, 1));
    int64_t p;
    for (p = 0; p < n; ++p) {
      int l;
      embed_rows(m, embed, tokens + off + p, 1, x);
      for (l = 0; l < m->num_layers; ++l) {
        const int kv_only = (l == m->num_layers - 1) && final_hidden == NULL;
        layer_step(m, &layers[l], l, x, p, 1, table, arena, kv_only, scratch);
      }
      if (final_hidden) memcpy(final_hidden + (off + p) * H, x, sizeof(double) * (size_t)H);
    }
    free(scratch);
    free(x);
    off += n;
  }
  return 0;
}

int kvo_decode_step(const kvo_model* m, const void* embed, const kvo_layer* layers,
                    const int32_t* tokens, const int32_t* positions, int32_t num_requests,
                    const int32_t* block_tables, int32_t max_blocks, kvo_arena* arena,
                    double* final_hidden) {
  int32_t r;
  if (!m || num_requests < 0 || !arena || !arena->base || arena->block_size <= 0) return -1;
  for (r = 0; r < num_requests; ++r) {
    const int64_t p = positions[r];
    int64_t b;
    if (p < 0 || p / arena->block_size >= max_blocks) return -1;
    if (tokens[r] < 0 || tokens[r] >= m->vocab) return -1;
    for (b = 0; b <= p / arena->block_size; ++b) {
      const int32_t blk = block_tables[(int64_t)r * max_blocks + b];
      if (blk < 0 || blk >= arena->num_blocks) return -1;
    }
  }
  for (r = 0; r < num_requests; ++r) {
    const int64_t H = m->hidden;
    const int32_t* table = block_tables + (int64_t)r * max_blocks;
    double* x = (double*)malloc(sizeof(double) * (size_t)H);
    double* scratch = (double*)malloc(sizeof(double) * scratch_elems(m, 1));
    int l;
    embed_rows(m, embed, tokens + r, 1, x);
    for (l = 0; l < m->num_layers; ++l) {
      const int kv_only = (l == m->num_layers - 1) && final_hidden == NULL;
      layer_step(m, &layers[l], l, x, positions[r], 1, table, arena, kv_only, scratch);
    }
    if (final_hidden) memcpy(final_hidden + (int64_t)r * H, x, sizeof(double) * (size_t)H);
    free(scratch);
    free(x);
  }
  return 0;
}

int kvo_logits(const kvo_model* m, const void* final_norm, const void* lm_head,
               const double* hidden, int64_t n, float* logits_out) {
  const int64_t H = m ? m->hidden : 0, V = m ? m->vocab : 0;
  double *a, *z;
  int64_t i;
  if (!m || !final_norm || !lm_head || !hidden || !logits_out || n < 0) return -1;
  a = (double*)malloc(sizeof(double) * (size_t)(n * H + 1));
  z = (double*)malloc(sizeof(double) * (size_t)(n * V + 1));
  rmsnorm(hidden, final_norm, m->dtype, H, m->rms_eps, n, a);
  project(lm_head, m->dtype, V, H, a, n, z);
  for (i = 0; i < n * V; ++i) logits_out[i] = (float)z[i];
  free(z);
  free(a);
  return 0;
}

int kvo_layer0_kv(const kvo_model* m, const void* embed, const kvo_layer* layer0,
                  const int32_t* tokens, const int32_t* positions, int64_t n, void* k_out,
                  void* v_out) {
  const int dt = m->dtype;
  const int64_t H = m->hidden, kvd = (int64_t)m->num_kv_heads * m->head_dim;
  int64_t i;
  if (!m || n < 0) return -1;
  for (i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= m->vocab || positions[i] < 0) return -1;
#pragma omp parallel for schedule(dynamic, 1)
  for (i = 0; i < n; ++i) {
    double* x = (double*)malloc(sizeof(double) * (size_t)(2 * H + 2 * kvd));
    double *a = x + H, *k = a + H, *v = k + kvd;
    int64_t r, e;
    embed_rows(m, embed, tokens + i, 1, x);
    {
      double ss = 0.0, inv;
      int64_t j;
      for (j = 0; j < H; ++j) ss += x[j] * x[j];
      inv = 1.0 / sqrt(ss / (double)H + m->rms_eps);
      for (j = 0; j < H; ++j) a[j] = rnd(load(layer0->attn_norm, dt, j) * x[j] * inv, dt);
    }
    for (r = 0; r < kvd; ++r) {
      k[r] = to_work(dot_row(layer0->wk, dt, r, H, a), dt);
      v[r] = to_work(dot_row(layer0->wv, dt, r, H, a), dt);
    }
    rope_row(k, m->num_kv_heads, m->head_dim, positions[i], m->rope_theta, dt);
    for (e = 0; e < kvd; ++e) {
      store(k_out, dt, i * kvd + e, rnd(k[e], dt));
      store(v_out, dt, i * kvd + e, rnd(v[e], dt));
    }
    free(x);
  }
  return 0;
}

int kvo_time_layers(const kvo_model* m, const void* embed, const kvo_layer* layers,
                    const int32_t* tokens, int32_t n, int32_t num_layers) {
  kvo_model mm = *m;
  kvo_arena ar;
  int32_t* table;
  int32_t nb, b;
  int rc;
  if (n <= 0 || num_layers <= 0 || num_layers > m->num_layers) return -1;
  mm.num_layers = num_layers;
  nb = (n + 15) / 16;
  table = (int32_t*)malloc(sizeof(int32_t) * (size_t)nb);
  for (b = 0; b < nb; ++b) table[b] = b;
  ar.block_size = 16;
  ar.num_blocks = nb;
  ar.base = calloc((size_t)num_layers * 2 * nb * 16 * m->num_kv_heads * m->head_dim,
                   m->dtype == KVO_F64 ? 8 : (m->dtype == KVO_F32 ? 4 : 2));
  {
    /* time full layers (attention and FFN included) by asking for the final hidden state */
    double* fh = (double*)malloc(sizeof(double) * (size_t)n * m->hidden);
    rc = kvo_rebuild(&mm, embed, layers, tokens, &n, 1, table, nb, &ar, fh);
    free(fh);
  }
  free(ar.base);
  free(table);
  return rc;
}

/* ------------------------------------------------------------------ */
/* commit digests of arena blocks (flush-free recovery)                */
/* ------------------------------------------------------------------ */
static int64_t elem_bytes(int dtype) { return dtype == KVO_F64 ? 8 : (dtype == KVO_F32 ? 4 : 2); }

uint64_t kvo_block_digest(const kvo_model* m, const kvo_arena* a, int64_t block, int32_t nslots,
                          int* ok) {
  const int64_t row = (int64_t)m->num_kv_heads * m->head_dim * elem_bytes(m->dtype);
  const uint8_t* base = (const uint8_t*)a->base;
  uint64_t sum = 0;
  uint32_t i = 0; /* word index, counted modulo 2^32 */
  int l, kv;
  int32_t s;
  int64_t w;
  *ok = -1;
  if (row % 4 != 0 || block < 0 || block >= a->num_blocks || nslots < 0 || nslots > a->block_size)
    return 0;
  for (l = 0; l < m->num_layers; ++l)
    for (kv = 0; kv < 2; ++kv)
      for (s = 0; s < nslots; ++s) {
        const int64_t slot = block * a->block_size + s;
        const uint8_t* p = base + arena_off(m, a, l, kv, slot) * elem_bytes(m->dtype);
        for (w = 0; w < row / 4; ++w, ++i) {
          const uint32_t u = (uint32_t)p[4 * w] | (uint32_t)p[4 * w + 1] << 8 |
                             (uint32_t)p[4 * w + 2] << 16 | (uint32_t)p[4 * w + 3] << 24;
          const uint32_t x = u ^ (uint32_t)(i * 0x9E3779B9u);
          sum += (uint64_t)x * (uint64_t)x;
        }
      }
  *ok = 0;
  return sum;
}

int kvo_verify(const kvo_model* m, const kvo_arena* a, const int32_t* lens, int32_t R,
               const int32_t* tables, int32_t max_blocks, const uint64_t* committed,
               uint64_t* digests, int32_t* intact) {
  const int32_t B = a->block_size;
  int64_t e = 0;
  int32_t r, j;
  if (!m || !a || !a->base || B <= 0 || R < 0 || !committed || !intact) return -1;
  for (r = 0; r < R; ++r) {
    const int32_t nb = (lens[r] + B - 1) / B;
    int leading = 1;
    if (lens[r] < 0 || nb > max_blocks) return -1;
    intact[r] = 0;
    for (j = 0; j < nb; ++j, ++e) {
      const int32_t n = lens[r] - j * B < B ? lens[r] - j * B : B;
      int ok;
      const uint64_t dg = kvo_block_digest(m, a, tables[(int64_t)r * max_blocks + j], n, &ok);
      if (ok != 0) return -1;
      if (digests) digests[e] = dg;
      if (leading && dg == committed[e]) intact[r] = j + 1;
      else leading = 0;
    }
  }
  return 0;
}
