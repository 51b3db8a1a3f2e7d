/*
 * CPU oracle for the multimodal speculative decoding (MSD) decode path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline of the benchmark may load this library; the product path never
 * does.  It shares no code with the HIP library.
 *
 * These are the numerical building blocks of a Llama-style decoder, written
 * as plain loops in float64.  Weights arrive as bfloat16 bit patterns and are
 * widened exactly.  Every dot product is summed sequentially over its inner
 * index in ascending order, one output element at a time, so a row's result
 * never depends on how many other rows are processed with it or on the thread
 * count; this is what makes the tree-versus-branch and speculative-versus-plain
 * invariants exact.  Threads only split independent output elements.
 *
 * The target forward follows the paper's preliminaries (Sec. 3.1, the MLLM
 * feature h and its projection head); the layer internals (pre-norm RMSNorm,
 * rotate-half RoPE, SwiGLU, grouped-query attention) are those of the Llama
 * family that LLaVA builds on.  The tree-masked attention follows the
 * tree-structured attention of the feature-level draft phase (Sec. 3.2).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static inline double bf16_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* Y[m][n] = sum_k X[m][k] * W[n][k]  (X: [M][K] f64, W: [N][K] bf16). */
void orc_linear(int M, int K, int N, const double* X, const uint16_t* W, double* Y) {
  double* XT = (double*)malloc(sizeof(double) * (size_t)K * (size_t)M);
  for (int m = 0; m < M; ++m)
    for (int k = 0; k < K; ++k) XT[(size_t)k * M + m] = X[(size_t)m * K + k];
#pragma omp parallel
  {
    double* acc = (double*)malloc(sizeof(double) * (size_t)M);
#pragma omp for schedule(static)
    for (int n = 0; n < N; ++n) {
      const uint16_t* w = W + (size_t)n * K;
      for (int m = 0; m < M; ++m) acc[m] = 0.0;
      for (int k = 0; k < K; ++k) {
        double wk = bf16_to_double(w[k]);
        const double* xk = XT + (size_t)k * M;
        for (int m = 0; m < M; ++m) acc[m] += xk[m] * wk;
      }
      for (int m = 0; m < M; ++m) Y[(size_t)m * N + n] = acc[m];
    }
    free(acc);
  }
  free(XT);
}

/* RMSNorm: Y = X / sqrt(mean(X^2) + eps) * g, row by row. */
void orc_rmsnorm(int M, int D, const double* X, const uint16_t* g, double eps, double* Y) {
  for (int m = 0; m < M; ++m) {
    const double* x = X + (size_t)m * D;
    double ss = 0.0;
    for (int i = 0; i < D; ++i) ss += x[i] * x[i];
    double r = 1.0 / sqrt(ss / D + eps);
    for (int i = 0; i < D; ++i) Y[(size_t)m * D + i] = x[i] * r * bf16_to_double(g[i]);
  }
}

/* Rotary embedding, rotate-half convention: within each head the pair
 * (x[i], x[i + hd/2]) is rotated by angle pos * theta^(-2i/hd). In place on
 * X: [M][n_heads * hd]. */
void orc_rope(int M, int n_heads, int hd, double* X, const int32_t* pos, double theta) {
  int half = hd / 2;
  for (int m = 0; m < M; ++m) {
    for (int i = 0; i < half; ++i) {
      double inv_freq = pow(theta, -2.0 * (double)i / (double)hd);
      double ang = (double)pos[m] * inv_freq;
      double c = cos(ang), s = sin(ang);
      for (int h = 0; h < n_heads; ++h) {
        double* x = X + (size_t)m * n_heads * hd + (size_t)h * hd;
        double a = x[i], b = x[i + half];
        x[i] = a * c - b * s;
        x[i + half] = b * c + a * s;
      }
    }
  }
}

/* SwiGLU gate: Y = silu(G) * U, silu(z) = z / (1 + exp(-z)). */
void orc_silu_mul(size_t n, const double* G, const double* U, double* Y) {
  for (size_t i = 0; i < n; ++i) Y[i] = G[i] / (1.0 + exp(-G[i])) * U[i];
}

/*
 * Attention of M query rows against one layer's cache.
 *   Q: [M][H*hd] (already rotated); Kc, Vc: [S][KV][hd] for this layer.
 *   Every query row sees all slots in [0, L).  Slots [L, L+R) form the
 *   "new" region: with anc == NULL the attention is causal and query row i
 *   sees region slot L+j for j <= i (then R == M); otherwise row i sees region
 *   slot L+j iff bit j of anc[i] is set (R <= 64).
 *   Head h reads kv head h / (H/KV).  Scores are scaled by 1/sqrt(hd) and
 *   normalised with the max subtracted; keys are visited in slot order.
 *   O: [M][H*hd].
 */
void orc_attention(int M, int H, int KV, int hd, const double* Q, const double* Kc,
                   const double* Vc, int L, int R, const uint64_t* anc, double* O) {
  int group = H / KV;
  double scale = 1.0 / sqrt((double)hd);
  int S = L + R;
#pragma omp parallel
  {
    double* p = (double*)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
    char* vis = (char*)malloc((size_t)(S > 0 ? S : 1));
#pragma omp for collapse(2) schedule(static)
    for (int i = 0; i < M; ++i) {
      for (int h = 0; h < H; ++h) {
        int g = h / group;
        const double* q = Q + (size_t)i * H * hd + (size_t)h * hd;
        double mx = -INFINITY;
        for (int s = 0; s < S; ++s) {
          int j = s - L;
          vis[s] = (s < L) || (anc ? (j < 64 && ((anc[i] >> j) & 1ULL)) : (j <= i));
          if (!vis[s]) continue;
          const double* k = Kc + ((size_t)s * KV + g) * hd;
          double dot = 0.0;
          for (int e = 0; e < hd; ++e) dot += q[e] * k[e];
          p[s] = dot * scale;
          if (p[s] > mx) mx = p[s];
        }
        double den = 0.0;
        for (int s = 0; s < S; ++s)
          if (vis[s]) {
            p[s] = exp(p[s] - mx);
            den += p[s];
          }
        double* o = O + (size_t)i * H * hd + (size_t)h * hd;
        for (int e = 0; e < hd; ++e) o[e] = 0.0;
        for (int s = 0; s < S; ++s) {
          if (!vis[s]) continue;
          const double* v = Vc + ((size_t)s * KV + g) * hd;
          double w = p[s] / den;
          for (int e = 0; e < hd; ++e) o[e] += w * v[e];
        }
      }
    }
    free(p);
    free(vis);
  }
}
