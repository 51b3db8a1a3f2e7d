// Kernels of the draft-head training step (Sec. 4.2) in float32: the
// teacher-forced draft layer over a training sequence, its loss (regression
// toward the next target feature plus the token cross-entropy against the
// target's next-token distribution) and the backward pass, and the AdamW
// update.  The contractions run as rocBLAS float32 GEMMs issued by the host
// orchestration; these kernels do everything between them.  Row-major
// throughout; a training pass has R = n - 1 rows (positions 0 .. n-2).
#include "msd_internal.h"

namespace msd {

namespace {

constexpr int TB = 256;

MSD_DEV float bsum(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  return (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

MSD_DEV float bmax(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  return fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3]));
}

// Row i < n: H[i] = target feature (split row hi + lo); for i < R also
// X0[i] = [h_i | e_{i+1}] and E0[i] = the draft input of a visual row i:
// e_i, or h_i with visual_feature (the Visual Feature variant), where e is
// the token embedding (text) or the visual row vis_idx (visual).  Grid (n),
// block TB.
__global__ __launch_bounds__(TB) void k_tr_inputs(const uint16_t* h, const uint16_t* E,
                                                  const int* tok, const int* vis_idx,
                                                  const uint16_t* visual, int n, int d,
                                                  int visual_feature, float* H, float* X0,
                                                  float* E0) {
  const int i = blockIdx.x;
  const int R = n - 1;
  const uint16_t* hr = h + (size_t)i * 2 * d;
  const int vi = vis_idx[i];
  const uint16_t* er = vi >= 0 ? visual + (size_t)vi * d : E + (size_t)tok[i] * d;
  for (int k = threadIdx.x; k < d; k += TB) {
    const float hv = bf2f(hr[k]) + bf2f(hr[d + k]);
    H[(size_t)i * d + k] = hv;
    if (i < R) {
      X0[(size_t)i * 2 * d + k] = hv;
      E0[(size_t)i * d + k] = visual_feature ? hv : bf2f(er[k]);
    }
    if (i > 0) X0[(size_t)(i - 1) * 2 * d + d + k] = bf2f(er[k]);
  }
}

// Visual rows take E0 as the draft input (Eq. decouple: their embedding, or
// their target feature in the Visual Feature variant).
__global__ __launch_bounds__(TB) void k_tr_visual_rows(float* F, const float* E0,
                                                       const int* vis_idx, int d) {
  const int i = blockIdx.x;
  if (vis_idx[i] < 0) return;
  for (int k = threadIdx.x; k < d; k += TB) F[(size_t)i * d + k] = E0[(size_t)i * d + k];
}

// Zeroes the rows of dF that are visual (they do not pass through f_down).
__global__ __launch_bounds__(TB) void k_tr_zero_visual(float* dF, const int* vis_idx, int d) {
  const int i = blockIdx.x;
  if (vis_idx[i] < 0) return;
  for (int k = threadIdx.x; k < d; k += TB) dF[(size_t)i * d + k] = 0.f;
}

// Y = x / sqrt(mean(x^2) + eps) * g, rstd[i] saved.  Grid (R).
__global__ __launch_bounds__(TB) void k_tr_rmsnorm(const float* X, const float* g, float eps,
                                                   int d, float* Y, float* rstd) {
  __shared__ float sh[4];
  const int i = blockIdx.x;
  const float* x = X + (size_t)i * d;
  float s = 0.f;
  for (int k = threadIdx.x; k < d; k += TB) s += x[k] * x[k];
  s = bsum(s, sh);
  const float r = rsqrtf(s / (float)d + eps);
  if (threadIdx.x == 0) rstd[i] = r;
  for (int k = threadIdx.x; k < d; k += TB) Y[(size_t)i * d + k] = x[k] * r * g[k];
}

// dX += the gradient of the RMSNorm input given dY (per row), with
// y = x r g, r = (mean(x^2) + eps)^-1/2: dx = r (g dy) - x r^3 mean(x g dy).
__global__ __launch_bounds__(TB) void k_tr_rmsnorm_bwd(const float* X, const float* g,
                                                       const float* rstd, const float* dY, int d,
                                                       float* dX) {
  __shared__ float sh[4];
  const int i = blockIdx.x;
  const float* x = X + (size_t)i * d;
  const float* dy = dY + (size_t)i * d;
  const float r = rstd[i];
  float s = 0.f;
  for (int k = threadIdx.x; k < d; k += TB) s += x[k] * g[k] * dy[k];
  s = bsum(s, sh) / (float)d;
  for (int k = threadIdx.x; k < d; k += TB)
    dX[(size_t)i * d + k] += r * g[k] * dy[k] - x[k] * r * r * r * s;
}

// dg[k] += sum over rows of dY[i][k] x[i][k] rstd[i] (a thread per feature,
// rows in order).
__global__ __launch_bounds__(TB) void k_tr_norm_gain_grad(const float* X, const float* rstd,
                                                          const float* dY, int R, int d,
                                                          float* dg) {
  const int k = blockIdx.x * TB + threadIdx.x;
  if (k >= d) return;
  float s = 0.f;
  for (int i = 0; i < R; ++i) s += dY[(size_t)i * d + k] * X[(size_t)i * d + k] * rstd[i];
  dg[k] += s;
}

// Rotate-half RoPE of X [R][nh*hd] at position = row, by +angle (dir 1) or
// -angle (dir -1, the backward of the forward rotation).  Grid (R, nh).
__global__ __launch_bounds__(TB) void k_tr_rope(float* X, int nh, int hd, const float2* tab,
                                                int dir) {
  const int i = blockIdx.x, h = blockIdx.y, half = hd / 2;
  float* x = X + ((size_t)i * nh + h) * hd;
  for (int k = threadIdx.x; k < half; k += TB) {
    const float2 t = tab[(size_t)i * half + k];
    const float c = t.x, s = dir > 0 ? t.y : -t.y;
    const float a = x[k], b = x[k + half];
    x[k] = a * c - b * s;
    x[k + half] = b * c + a * s;
  }
}

// Causal softmax of S [R][R] rows (one head): P[i][j] = softmax_j<=i(scale
// S[i][j]), 0 above the diagonal.  Grid (R, heads); S in place.
__global__ __launch_bounds__(TB) void k_tr_softmax(float* S, int R, float scale) {
  __shared__ float sh[4];
  const int i = blockIdx.x;
  float* s = S + ((size_t)blockIdx.y * R + i) * R;
  float m = -INFINITY;
  for (int j = threadIdx.x; j <= i; j += TB) m = fmaxf(m, s[j] * scale);
  m = bmax(m, sh);
  float z = 0.f;
  for (int j = threadIdx.x; j <= i; j += TB) z += __expf(s[j] * scale - m);
  z = bsum(z, sh);
  const float inv = 1.f / z;
  for (int j = threadIdx.x; j < R; j += TB) s[j] = j <= i ? __expf(s[j] * scale - m) * inv : 0.f;
}

// dS = scale P (dP - rowsum(dP P)), in place over dP.  Grid (R, heads).
__global__ __launch_bounds__(TB) void k_tr_softmax_bwd(const float* P, float* dP, int R,
                                                       float scale) {
  __shared__ float sh[4];
  const size_t o = ((size_t)blockIdx.y * R + blockIdx.x) * R;
  float t = 0.f;
  for (int j = threadIdx.x; j < R; j += TB) t += dP[o + j] * P[o + j];
  t = bsum(t, sh);
  for (int j = threadIdx.x; j < R; j += TB) dP[o + j] = scale * P[o + j] * (dP[o + j] - t);
}

// Mx = silu(G) * U, n elements.
__global__ __launch_bounds__(TB) void k_tr_silu(const float* G, const float* U, size_t n,
                                                float* Mx) {
  const size_t k = (size_t)blockIdx.x * TB + threadIdx.x;
  if (k >= n) return;
  const float g = G[k];
  Mx[k] = g / (1.f + __expf(-g)) * U[k];
}

// dG = dM U silu'(G), dU = dM silu(G) (silu' = s (1 + g (1 - s)), s = sigmoid).
__global__ __launch_bounds__(TB) void k_tr_silu_bwd(const float* G, const float* U,
                                                    const float* dM, size_t n, float* dG,
                                                    float* dU) {
  const size_t k = (size_t)blockIdx.x * TB + threadIdx.x;
  if (k >= n) return;
  const float g = G[k], s = 1.f / (1.f + __expf(-g));
  dG[k] = dM[k] * U[k] * s * (1.f + g * (1.f - s));
  dU[k] = dM[k] * g * s;
}

// Regression term of row i: sum over features of SmoothL1(D[i] - H[i+1])
// divided by d into reg[i], its gradient into dD.  Grid (R).
__global__ __launch_bounds__(TB) void k_tr_reg(const float* D, const float* H, int d,
                                               float* dD, float* reg) {
  __shared__ float sh[4];
  const int i = blockIdx.x;
  float s = 0.f;
  for (int k = threadIdx.x; k < d; k += TB) {
    const float x = D[(size_t)i * d + k] - H[(size_t)(i + 1) * d + k];
    const float a = fabsf(x);
    s += a < 1.f ? 0.5f * x * x : a - 0.5f;
    dD[(size_t)i * d + k] = fminf(fmaxf(x, -1.f), 1.f) / (float)d;
  }
  s = bsum(s, sh);
  if (threadIdx.x == 0) reg[i] = s / (float)d;
}

// Token term of row i: with p = softmax(Ld[i]) (draft) and q =
// softmax(Lt[i]) (target, the row of position i + 1), ce[i] = -sum q log p,
// and Ld[i] <- w (p - q), the gradient of w ce[i].  Grid (R).
__global__ __launch_bounds__(TB) void k_tr_ce(float* Ld, const float* Lt, int V, float w,
                                              float* ce) {
  __shared__ float sh[4];
  float* ld = Ld + (size_t)blockIdx.x * V;
  const float* lt = Lt + (size_t)blockIdx.x * V;
  float md = -INFINITY, mt = -INFINITY;
  for (int v = threadIdx.x; v < V; v += TB) {
    md = fmaxf(md, ld[v]);
    mt = fmaxf(mt, lt[v]);
  }
  md = bmax(md, sh);
  mt = bmax(mt, sh);
  float zd = 0.f, zt = 0.f;
  for (int v = threadIdx.x; v < V; v += TB) {
    zd += __expf(ld[v] - md);
    zt += __expf(lt[v] - mt);
  }
  zd = bsum(zd, sh);
  zt = bsum(zt, sh);
  const float lzd = logf(zd);
  float c = 0.f;
  for (int v = threadIdx.x; v < V; v += TB) {
    const float q = __expf(lt[v] - mt) / zt;
    const float lp = ld[v] - md - lzd;
    c -= q * lp;
    ld[v] = w * (__expf(lp) - q);
  }
  c = bsum(c, sh);
  if (threadIdx.x == 0) ce[blockIdx.x] = c;
}

// w -= lr mhat / (sqrt(vhat) + eps) with g = gsum * gscale (AdamW, no decay),
// and the bfloat16 copy of the new w (round to nearest even).
__global__ __launch_bounds__(TB) void k_tr_adamw(float* w, const float* gsum, float* m, float* v,
                                                 size_t n, float gscale, float lr, float c1,
                                                 float c2, float b1, float b2, float eps,
                                                 uint16_t* wb) {
  const size_t k = (size_t)blockIdx.x * TB + threadIdx.x;
  if (k >= n) return;
  const float g = gsum[k] * gscale;
  const float mk = b1 * m[k] + (1.f - b1) * g;
  const float vk = b2 * v[k] + (1.f - b2) * g * g;
  m[k] = mk;
  v[k] = vk;
  const float wk = w[k] - lr * (mk / c1) / (sqrtf(vk / c2) + eps);
  w[k] = wk;
  wb[k] = f2bf(wk);
}

__global__ __launch_bounds__(TB) void k_tr_widen(const uint16_t* src, size_t n, float* dst) {
  const size_t k = (size_t)blockIdx.x * TB + threadIdx.x;
  if (k < n) dst[k] = bf2f(src[k]);
}

__global__ __launch_bounds__(TB) void k_tr_fill(float* p, size_t n, float v) {
  const size_t k = (size_t)blockIdx.x * TB + threadIdx.x;
  if (k < n) p[k] = v;
}

unsigned blocks(size_t n) { return (unsigned)((n + TB - 1) / TB); }

}  // namespace

void tr_inputs(const uint16_t* h, const uint16_t* E, const int* tok, const int* vis_idx,
               const uint16_t* visual, int n, int d, int visual_feature, float* H, float* X0,
               float* E0, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_inputs, dim3(n), dim3(TB), 0, st, h, E, tok, vis_idx, visual, n, d,
                     visual_feature, H, X0, E0);
}
void tr_visual_rows(float* F, const float* E0, const int* vis_idx, int R, int d, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_visual_rows, dim3(R), dim3(TB), 0, st, F, E0, vis_idx, d);
}
void tr_zero_visual(float* dF, const int* vis_idx, int R, int d, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_zero_visual, dim3(R), dim3(TB), 0, st, dF, vis_idx, d);
}
void tr_rmsnorm(const float* X, const float* g, float eps, int R, int d, float* Y, float* rstd,
                hipStream_t st) {
  hipLaunchKernelGGL(k_tr_rmsnorm, dim3(R), dim3(TB), 0, st, X, g, eps, d, Y, rstd);
}
void tr_rmsnorm_bwd(const float* X, const float* g, const float* rstd, const float* dY, int R,
                    int d, float* dX, float* dg, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_rmsnorm_bwd, dim3(R), dim3(TB), 0, st, X, g, rstd, dY, d, dX);
  hipLaunchKernelGGL(k_tr_norm_gain_grad, dim3(blocks(d)), dim3(TB), 0, st, X, rstd, dY, R, d, dg);
}
void tr_rope(float* X, int R, int nh, int hd, const float2* tab, int dir, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_rope, dim3(R, nh), dim3(TB), 0, st, X, nh, hd, tab, dir);
}
void tr_softmax(float* S, int R, int heads, float scale, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_softmax, dim3(R, heads), dim3(TB), 0, st, S, R, scale);
}
void tr_softmax_bwd(const float* P, float* dP, int R, int heads, float scale, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_softmax_bwd, dim3(R, heads), dim3(TB), 0, st, P, dP, R, scale);
}
void tr_silu(const float* G, const float* U, size_t n, float* Mx, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_silu, dim3(blocks(n)), dim3(TB), 0, st, G, U, n, Mx);
}
void tr_silu_bwd(const float* G, const float* U, const float* dM, size_t n, float* dG, float* dU,
                 hipStream_t st) {
  hipLaunchKernelGGL(k_tr_silu_bwd, dim3(blocks(n)), dim3(TB), 0, st, G, U, dM, n, dG, dU);
}
void tr_reg(const float* D, const float* H, int R, int d, float* dD, float* reg, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_reg, dim3(R), dim3(TB), 0, st, D, H, d, dD, reg);
}
void tr_ce(float* Ld, const float* Lt, int R, int V, float w, float* ce, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_ce, dim3(R), dim3(TB), 0, st, Ld, Lt, V, w, ce);
}
void tr_adamw(float* w, const float* gsum, float* m, float* v, size_t n, float gscale, float lr,
              float c1, float c2, float b1, float b2, float eps, uint16_t* wb, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_adamw, dim3(blocks(n)), dim3(TB), 0, st, w, gsum, m, v, n, gscale, lr,
                     c1, c2, b1, b2, eps, wb);
}
void tr_widen(const uint16_t* src, size_t n, float* dst, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_widen, dim3(blocks(n)), dim3(TB), 0, st, src, n, dst);
}
void tr_fill(float* p, size_t n, float v, hipStream_t st) {
  hipLaunchKernelGGL(k_tr_fill, dim3(blocks(n)), dim3(TB), 0, st, p, n, v);
}

}  // namespace msd
