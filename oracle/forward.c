/* Oracle: the window forward of a LLaMA-style decoder (ParallelForward of
 * Alg. 1): every window slot is evaluated in one pass over the cached keys
 * and values plus the window itself.
 *
 * Test infrastructure only (see oracle.h); shares no code with the HIP path.
 *
 * The paper names its models (Lumina-mGPT 7B, Emu3 8B; Sec. 5.1) but not
 * their layers; the layer used here is the usual pre-norm decoder block:
 *   h = x + Wo . Attn(RoPE(Wq . n1(x)), RoPE(Wk . n1(x)), Wv . n1(x))
 *   x' = h + Wd . (silu(Wg . n2(h)) * (Wu . n2(h)))
 * with RMS norms n(x) = x / sqrt(mean(x^2) + eps) * g, rotary embeddings in
 * the rotate-half layout (pair i with i + hd/2, angle pos * theta^(-2i/hd)),
 * grouped-query attention (query head h reads key/value head h / (H / Hkv)),
 * scale 1 / sqrt(hd), and an untied head restricted to the rows of the
 * sampled vocabulary range.
 *
 * Masking follows the tree of the window: slot a sees every cached row and
 * the window slots whose bit is set in anc[a] (its ancestors and itself).
 *
 * Arithmetic: bf16 weights are widened exactly to fp32; every dot product
 * and reduction accumulates in fp64; activations and the cache are kept in
 * fp64. This is deliberately plain and slow.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

struct orc_kv {
  orc_model_cfg cfg;
  double* k; /* [layers][max_seq][Hkv*hd] */
  double* v; /* [layers][max_seq][Hkv*hd] */
};

orc_kv* orc_kv_new(const orc_model_cfg* cfg) {
  orc_kv* kv = (orc_kv*)calloc(1, sizeof(orc_kv));
  if (!kv) return NULL;
  kv->cfg = *cfg;
  size_t n = (size_t)cfg->n_layers * cfg->max_seq * cfg->n_kv_heads * cfg->head_dim;
  kv->k = (double*)calloc(n, sizeof(double));
  kv->v = (double*)calloc(n, sizeof(double));
  if (!kv->k || !kv->v) { orc_kv_free(kv); return NULL; }
  return kv;
}

void orc_kv_free(orc_kv* kv) {
  if (!kv) return;
  free(kv->k);
  free(kv->v);
  free(kv);
}

void orc_kv_move(orc_kv* kv, int src, int dst) {
  const orc_model_cfg* c = &kv->cfg;
  size_t row = (size_t)c->n_kv_heads * c->head_dim;
  for (int l = 0; l < c->n_layers; ++l) {
    size_t base = (size_t)l * c->max_seq * row;
    memmove(kv->k + base + (size_t)dst * row, kv->k + base + (size_t)src * row, row * sizeof(double));
    memmove(kv->v + base + (size_t)dst * row, kv->v + base + (size_t)src * row, row * sizeof(double));
  }
}

void orc_kv_row(const orc_kv* kv, int layer, int row, double* k, double* v) {
  const orc_model_cfg* c = &kv->cfg;
  size_t n = (size_t)c->n_kv_heads * c->head_dim;
  size_t off = ((size_t)layer * c->max_seq + (size_t)row) * n;
  memcpy(k, kv->k + off, n * sizeof(double));
  memcpy(v, kv->v + off, n * sizeof(double));
}

static inline float bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* element i of a weight array */
static inline double wget(const void* base, int is_f32, size_t i) {
  if (is_f32) return (double)((const float*)base)[i];
  return (double)bf16_to_f32(((const uint16_t*)base)[i]);
}

/* y[a][o] = sum_i W[row0 + o][i] * x[a][i] for a < M, o < n_out; W has n_in columns. */
static void linear(const void* W, int is_f32, size_t row0, int n_out, int n_in, const double* x, int M,
                   double* y) {
#pragma omp parallel
  {
    double* wrow = (double*)malloc(sizeof(double) * (size_t)n_in);
#pragma omp for schedule(static)
    for (int o = 0; o < n_out; ++o) {
      size_t off = (row0 + (size_t)o) * (size_t)n_in;
      for (int i = 0; i < n_in; ++i) wrow[i] = wget(W, is_f32, off + (size_t)i);
      for (int a = 0; a < M; ++a) {
        const double* xa = x + (size_t)a * n_in;
        double s = 0.0;
        for (int i = 0; i < n_in; ++i) s += wrow[i] * xa[i];
        y[(size_t)a * n_out + o] = s;
      }
    }
    free(wrow);
  }
}

static void rmsnorm(const double* x, const void* g, int is_f32, int M, int d, double eps, double* y) {
  for (int a = 0; a < M; ++a) {
    const double* xa = x + (size_t)a * d;
    double ss = 0.0;
    for (int i = 0; i < d; ++i) ss += xa[i] * xa[i];
    double inv = 1.0 / sqrt(ss / d + eps);
    for (int i = 0; i < d; ++i) y[(size_t)a * d + i] = xa[i] * inv * wget(g, is_f32, (size_t)i);
  }
}

/* rotate-half rotary embedding of one head vector in place */
static void rope(double* v, int hd, int pos, double theta) {
  int half = hd / 2;
  for (int i = 0; i < half; ++i) {
    double freq = pow(theta, -2.0 * i / hd);
    double ang = (double)pos * freq;
    double cs = cos(ang), sn = sin(ang);
    double a = v[i], b = v[i + half];
    v[i] = a * cs - b * sn;
    v[i + half] = a * sn + b * cs;
  }
}

int orc_forward(const orc_model_cfg* c, const orc_weights* w, orc_kv* kv, int n,
                const int32_t* tok, const int32_t* pos, const uint64_t* anc, int M,
                float* logits) {
  const int d = c->d_model, H = c->n_heads, Hkv = c->n_kv_heads, hd = c->head_dim, F = c->ffn_dim;
  if (M < 1 || M > 64 || n < 0 || n + M > c->max_seq || H % Hkv != 0 || hd % 2 != 0) return -1;
  for (int a = 0; a < M; ++a) {
    if (tok[a] < 0 || tok[a] >= c->vocab_size) return -1;
    if (!((anc[a] >> a) & 1u)) return -1;
  }
  const int f32 = w->is_f32;
  const int qd = H * hd, kvd = Hkv * hd;
  const size_t kvrow = (size_t)kvd;
  double* x = (double*)malloc(sizeof(double) * (size_t)M * d);
  double* xn = (double*)malloc(sizeof(double) * (size_t)M * d);
  double* q = (double*)malloc(sizeof(double) * (size_t)M * qd);
  double* kk = (double*)malloc(sizeof(double) * (size_t)M * kvd);
  double* vv = (double*)malloc(sizeof(double) * (size_t)M * kvd);
  double* att = (double*)malloc(sizeof(double) * (size_t)M * qd);
  double* tmp = (double*)malloc(sizeof(double) * (size_t)M * (d > F ? d : F));
  double* g = (double*)malloc(sizeof(double) * (size_t)M * F);
  double* u = (double*)malloc(sizeof(double) * (size_t)M * F);
  if (!x || !xn || !q || !kk || !vv || !att || !tmp || !g || !u) {
    free(x); free(xn); free(q); free(kk); free(vv); free(att); free(tmp); free(g); free(u);
    return -2;
  }
  for (int a = 0; a < M; ++a)
    for (int i = 0; i < d; ++i) x[(size_t)a * d + i] = wget(w->embed, f32, (size_t)tok[a] * d + i);

  const double scale = 1.0 / sqrt((double)hd);
  const int group = H / Hkv;
  for (int l = 0; l < c->n_layers; ++l) {
    const void* const* lw = w->layer + (size_t)l * 9;
    double* Kc = kv->k + (size_t)l * c->max_seq * kvrow;
    double* Vc = kv->v + (size_t)l * c->max_seq * kvrow;
    rmsnorm(x, lw[0], f32, M, d, c->rms_eps, xn);
    linear(lw[1], f32, 0, qd, d, xn, M, q);
    linear(lw[2], f32, 0, kvd, d, xn, M, kk);
    linear(lw[3], f32, 0, kvd, d, xn, M, vv);
    for (int a = 0; a < M; ++a) {
      for (int h = 0; h < H; ++h) rope(q + (size_t)a * qd + (size_t)h * hd, hd, pos[a], c->rope_theta);
      for (int h = 0; h < Hkv; ++h) rope(kk + (size_t)a * kvd + (size_t)h * hd, hd, pos[a], c->rope_theta);
      memcpy(Kc + (size_t)(n + a) * kvrow, kk + (size_t)a * kvd, sizeof(double) * kvrow);
      memcpy(Vc + (size_t)(n + a) * kvrow, vv + (size_t)a * kvd, sizeof(double) * kvrow);
    }
#pragma omp parallel for collapse(2) schedule(static)
    for (int a = 0; a < M; ++a) {
      for (int h = 0; h < H; ++h) {
        const int hk = h / group;
        const double* qa = q + (size_t)a * qd + (size_t)h * hd;
        int nk = n + M;
        double* sc = (double*)malloc(sizeof(double) * (size_t)nk);
        double mx = -INFINITY;
        for (int t = 0; t < nk; ++t) {
          int vis = t < n || ((anc[a] >> (t - n)) & 1u);
          if (!vis) { sc[t] = -INFINITY; continue; }
          const double* kt = Kc + (size_t)t * kvrow + (size_t)hk * hd;
          double s = 0.0;
          for (int i = 0; i < hd; ++i) s += qa[i] * kt[i];
          sc[t] = s * scale;
          if (sc[t] > mx) mx = sc[t];
        }
        double Z = 0.0;
        for (int t = 0; t < nk; ++t) {
          sc[t] = (sc[t] == -INFINITY) ? 0.0 : exp(sc[t] - mx);
          Z += sc[t];
        }
        double* oa = att + (size_t)a * qd + (size_t)h * hd;
        for (int i = 0; i < hd; ++i) oa[i] = 0.0;
        for (int t = 0; t < nk; ++t) {
          if (sc[t] == 0.0) continue;
          const double* vt = Vc + (size_t)t * kvrow + (size_t)hk * hd;
          double pw = sc[t] / Z;
          for (int i = 0; i < hd; ++i) oa[i] += pw * vt[i];
        }
        free(sc);
      }
    }
    linear(lw[4], f32, 0, d, qd, att, M, tmp);
    for (size_t i = 0; i < (size_t)M * d; ++i) x[i] += tmp[i];
    rmsnorm(x, lw[5], f32, M, d, c->rms_eps, xn);
    linear(lw[6], f32, 0, F, d, xn, M, g);
    linear(lw[7], f32, 0, F, d, xn, M, u);
    for (size_t i = 0; i < (size_t)M * F; ++i) {
      double gi = g[i];
      g[i] = gi / (1.0 + exp(-gi)) * u[i];
    }
    linear(lw[8], f32, 0, d, F, g, M, tmp);
    for (size_t i = 0; i < (size_t)M * d; ++i) x[i] += tmp[i];
  }
  if (logits) {
    rmsnorm(x, w->final_norm, f32, M, d, c->rms_eps, xn);
    double* lg = (double*)malloc(sizeof(double) * (size_t)M * c->V);
    if (!lg) { free(x); free(xn); free(q); free(kk); free(vv); free(att); free(tmp); free(g); free(u); return -2; }
    linear(w->lm_head, f32, (size_t)c->vis_lo, c->V, d, xn, M, lg);
    for (size_t i = 0; i < (size_t)M * c->V; ++i) logits[i] = (float)lg[i];
    free(lg);
  }
  free(x); free(xn); free(q); free(kk); free(vv); free(att); free(tmp); free(g); free(u);
  return 0;
}

/* Classifier-free guidance (Sec. 5.1): l = l_u + w (l_c - l_u), fp64. */
void orc_cfg_combine(const float* l_c, const float* l_u, float w, long n, float* out) {
  for (long i = 0; i < n; ++i) out[i] = (float)((double)l_u[i] + (double)w * ((double)l_c[i] - (double)l_u[i]));
}

