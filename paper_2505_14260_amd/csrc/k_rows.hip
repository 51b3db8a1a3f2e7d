// Row-wise kernels of the decode path: embedding gather, RMSNorm, rotary
// embedding with the KV-cache write, the draft input builder and the
// vocabulary top-k / logsumexp.
#include "msd_internal.h"

namespace msd {

namespace {

// Block-wide sum over 256 threads in a fixed order (deterministic).
MSD_DEV float block_sum_256(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  return (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

// x[row] = E[token] (text) or visual[vis_idx] (visual rows), widened to f32.
__global__ __launch_bounds__(256) void k_embed(const uint16_t* E, const int* tokens,
                                               const int* vis_idx, const uint16_t* visual,
                                               int d, float* x) {
  const int row = blockIdx.x;
  const int v = vis_idx ? vis_idx[row] : -1;
  const uint16_t* src = (v >= 0) ? visual + (size_t)v * d : E + (size_t)tokens[row] * d;
  // token ids were validated on the host or clamped by the row builder
  float* dst = x + (size_t)row * d;
  for (int e = threadIdx.x; e < d; e += 256) dst[e] = bf2f(src[e]);
}

// Overwrites the visual rows of x with their embeddings (draft input rule for
// visual positions: the embedding itself, no down-projection).
__global__ __launch_bounds__(256) void k_visual_rows(const uint16_t* visual, const int* vis_idx,
                                                     int d, float* x) {
  const int row = blockIdx.x;
  const int v = vis_idx[row];
  if (v < 0) return;
  for (int e = threadIdx.x; e < d; e += 256) x[(size_t)row * d + e] = bf2f(visual[(size_t)v * d + e]);
}

// y = bf16(x / sqrt(mean(x^2) + eps) * g)
__global__ __launch_bounds__(256) void k_rmsnorm(const float* x, const uint16_t* g, int d,
                                                 float eps, uint16_t* y) {
  __shared__ float sh[4];
  const int row = blockIdx.x;
  const float* xr = x + (size_t)row * d;
  float ss = 0.f;
  for (int e = threadIdx.x; e < d; e += 256) ss += xr[e] * xr[e];
  ss = block_sum_256(ss, sh);
  const float r = rsqrtf(ss / (float)d + eps);
  for (int e = threadIdx.x; e < d; e += 256) y[(size_t)row * d + e] = f2bf(xr[e] * r * bf2f(g[e]));
}

__global__ void k_to_bf16(const float* x, int n, uint16_t* y) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = f2bf(x[i]);
}

// cos/sin of pos * theta^(-2i/hd), evaluated in float64.
__global__ void k_rope_table(float2* tab, int max_pos, int half, double theta) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= max_pos * half) return;
  const int pos = idx / half, i = idx - pos * half;
  const double inv = pow(theta, -2.0 * (double)i / (double)(2 * half));
  double s, c;
  sincos((double)pos * inv, &s, &c);
  tab[idx] = make_float2((float)c, (float)s);
}

// Rotate-half RoPE on q and k, write q (bf16), K to its slot and V to the
// transposed V cache.  qkv: [rows][(H + 2KV) * hd] f32.
__global__ __launch_bounds__(256) void k_rope_kv(const float* qkv, int H, int KV, int hd,
                                                 const int* pos, const int* row_seq,
                                                 const int* row_slot, const float2* tab,
                                                 uint16_t* q, uint16_t* kc, uint16_t* vc, int S) {
  const int row = blockIdx.x;
  const int half = hd / 2;
  const int ld = (H + 2 * KV) * hd;
  const float* src = qkv + (size_t)row * ld;
  const float2* cs = tab + (size_t)pos[row] * half;
  const int slot = row_slot[row];
  const int b = row_seq[row];
  for (int idx = threadIdx.x; idx < (H + KV) * half; idx += 256) {
    const int head = idx / half, i = idx - head * half;
    const float* x = src + head * hd;
    const float a = x[i], c = x[i + half];
    const float2 t = cs[i];
    const float y0 = a * t.x - c * t.y;
    const float y1 = c * t.x + a * t.y;
    if (head < H) {
      q[(size_t)row * H * hd + head * hd + i] = f2bf(y0);
      q[(size_t)row * H * hd + head * hd + i + half] = f2bf(y1);
    } else if (slot >= 0) {
      const int g = head - H;
      uint16_t* kr = kc + ((size_t)(b * KV + g) * S + slot) * hd;
      kr[i] = f2bf(y0);
      kr[i + half] = f2bf(y1);
    }
  }
  if (slot < 0) return;
  for (int idx = threadIdx.x; idx < KV * hd; idx += 256) {
    const int g = idx / hd, e = idx - g * hd;
    vc[((size_t)(b * KV + g) * hd + e) * S + slot] = f2bf(src[(H + KV) * hd + idx]);
  }
}

// out[row] = [h_row | e_next] in bf16, the concat fed to the draft's f_down.
// h comes from bf16 rows (target features) or f32 rows (draft features);
// next_tok >= 0 selects E[next_tok], next_tok < 0 selects visual row -1-next_tok.
__global__ __launch_bounds__(256) void k_fc_input(const uint16_t* h, const float* hf,
                                                  const int* h_row, const uint16_t* E,
                                                  const int* next_tok, const uint16_t* visual,
                                                  int d, uint16_t* out) {
  const int row = blockIdx.x;
  const int hr = h_row[row];
  const int nt = next_tok[row];
  const uint16_t* e = (nt >= 0) ? E + (size_t)nt * d : visual + (size_t)(-1 - nt) * d;
  uint16_t* o = out + (size_t)row * 2 * d;
  for (int i = threadIdx.x; i < d; i += 256) {
    o[i] = h ? h[(size_t)hr * d + i] : f2bf(hf[(size_t)hr * d + i]);
    o[d + i] = e[i];
  }
}

// Per-row top-k over the vocabulary (value descending, then id ascending)
// and the row's logsumexp, in two phases: every (row, slice) block reduces a
// slice of the vocabulary to its own top-k and (max, sum of exp) pair; one
// block per row then merges the slices in slice order.
constexpr int TOPK_MAX = 16;
constexpr int TOPK_SLICE = 2048;

MSD_DEV bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// Block-wide selection of the k best (value, id) pairs offered by each
// thread's sorted local list (lv, li of length n).
MSD_DEV void block_select(const float* lv, const int* li, int n, int k, float* sv, int* si,
                          float* out_v, int* out_i) {
  int head = 0;
  for (int q = 0; q < k; ++q) {
    sv[threadIdx.x] = (head < n) ? lv[head] : -INFINITY;
    si[threadIdx.x] = (head < n) ? li[head] : 0x7FFFFFFF;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
      if (threadIdx.x < s) {
        const float vb = sv[threadIdx.x + s];
        const int ib = si[threadIdx.x + s];
        if (better(vb, ib, sv[threadIdx.x], si[threadIdx.x])) {
          sv[threadIdx.x] = vb;
          si[threadIdx.x] = ib;
        }
      }
      __syncthreads();
    }
    const int win = si[0];
    const float wv = sv[0];
    __syncthreads();
    if (head < n && li[head] == win) ++head;
    if (threadIdx.x == 0) {
      out_i[q] = win;
      out_v[q] = wv;
    }
  }
}

MSD_DEV void insert_sorted(float* lv, int* li, int& n, int k, float val, int id) {
  if (n < k || better(val, id, lv[k - 1], li[k - 1])) {
    int p = (n < k) ? n : k - 1;
    while (p > 0 && better(val, id, lv[p - 1], li[p - 1])) {
      lv[p] = lv[p - 1];
      li[p] = li[p - 1];
      --p;
    }
    lv[p] = val;
    li[p] = id;
    if (n < k) ++n;
  }
}

__global__ __launch_bounds__(256) void k_topk_slice(const float* logits, int V, int k, int n_slices,
                                                    float* cand_v, int* cand_i, float2* stats) {
  __shared__ float sv[256];
  __shared__ int si[256];
  __shared__ float sm[4];
  __shared__ float ssum[4];
  const int row = blockIdx.x / n_slices;
  const int sl = blockIdx.x - row * n_slices;
  const float* x = logits + (size_t)row * V;
  const int v0 = sl * TOPK_SLICE, v1 = min(V, v0 + TOPK_SLICE);
  float lv[TOPK_MAX];
  int li[TOPK_MAX];
  int n = 0;
  float mloc = -INFINITY, sloc = 0.f;
  for (int v = v0 + threadIdx.x; v < v1; v += 256) {
    const float val = x[v];
    if (val > mloc) {
      sloc = sloc * __expf(mloc - val) + 1.f;
      mloc = val;
    } else {
      sloc += __expf(val - mloc);
    }
    insert_sorted(lv, li, n, k, val, v);
  }
  float mm = mloc;
  for (int o = 32; o > 0; o >>= 1) mm = fmaxf(mm, __shfl_xor(mm, o));
  if ((threadIdx.x & 63) == 0) sm[threadIdx.x >> 6] = mm;
  __syncthreads();
  const float M = fmaxf(fmaxf(sm[0], sm[1]), fmaxf(sm[2], sm[3]));
  const float part = (mloc == -INFINITY) ? 0.f : sloc * __expf(mloc - M);
  const float tot = block_sum_256(part, ssum);
  if (threadIdx.x == 0) stats[blockIdx.x] = make_float2(M, tot);
  block_select(lv, li, n, k, sv, si, cand_v + (size_t)blockIdx.x * k,
               cand_i + (size_t)blockIdx.x * k);
}

__global__ __launch_bounds__(256) void k_topk_merge(int k, int n_slices, const float* cand_v,
                                                    const int* cand_i, const float2* stats,
                                                    int* out_idx, float* out_val, float* out_lse) {
  __shared__ float sv[256];
  __shared__ int si[256];
  __shared__ float ov[TOPK_MAX];
  __shared__ int oi[TOPK_MAX];
  const int row = blockIdx.x;
  const size_t c0 = (size_t)row * n_slices * k;
  float lv[TOPK_MAX];
  int li[TOPK_MAX];
  int n = 0;
  for (int c = threadIdx.x; c < n_slices * k; c += 256)
    insert_sorted(lv, li, n, k, cand_v[c0 + c], cand_i[c0 + c]);
  block_select(lv, li, n, k, sv, si, ov, oi);
  __syncthreads();
  if (threadIdx.x < k) {
    out_idx[(size_t)row * k + threadIdx.x] = oi[threadIdx.x];
    if (out_val) out_val[(size_t)row * k + threadIdx.x] = ov[threadIdx.x];
  }
  if (threadIdx.x == 0 && out_lse) {
    const float2* st = stats + (size_t)row * n_slices;
    float M = -INFINITY;
    for (int q = 0; q < n_slices; ++q) M = fmaxf(M, st[q].x);
    float tot = 0.f;
    for (int q = 0; q < n_slices; ++q)
      tot += (st[q].x == -INFINITY) ? 0.f : st[q].y * __expf(st[q].x - M);
    out_lse[row] = M + __logf(tot);
  }
}

}  // namespace

void launch_embed(const uint16_t* E, const int* tokens, const int* vis_idx,
                  const uint16_t* visual, int rows, int d, float* x, hipStream_t st) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_embed, dim3(rows), dim3(256), 0, st, E, tokens, vis_idx, visual, d, x);
}

void launch_visual_rows(const uint16_t* visual, const int* vis_idx, int rows, int d, float* x,
                        hipStream_t st) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_visual_rows, dim3(rows), dim3(256), 0, st, visual, vis_idx, d, x);
}

void launch_rmsnorm(const float* x, const uint16_t* g, int rows, int d, float eps, uint16_t* y,
                    hipStream_t st) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_rmsnorm, dim3(rows), dim3(256), 0, st, x, g, d, eps, y);
}

void launch_to_bf16(const float* x, int n, uint16_t* y, hipStream_t st) {
  if (n <= 0) return;
  hipLaunchKernelGGL(k_to_bf16, dim3((n + 255) / 256), dim3(256), 0, st, x, n, y);
}

void launch_rope_table(float2* tab, int max_pos, int hd, double theta, hipStream_t st) {
  const int n = max_pos * (hd / 2);
  hipLaunchKernelGGL(k_rope_table, dim3((n + 255) / 256), dim3(256), 0, st, tab, max_pos,
                     hd / 2, theta);
}

void launch_rope_kv(const float* qkv, int rows, int H, int KV, int hd, const int* pos,
                    const int* row_seq, const int* row_slot, const float2* rope_tab,
                    uint16_t* q, uint16_t* kc, uint16_t* vc, int S, hipStream_t st) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_rope_kv, dim3(rows), dim3(256), 0, st, qkv, H, KV, hd, pos, row_seq,
                     row_slot, rope_tab, q, kc, vc, S);
}

void launch_fc_input(const uint16_t* h, const float* hf, const int* h_row, const uint16_t* E,
                     const int* next_tok, const uint16_t* visual, int rows, int d,
                     uint16_t* out, hipStream_t st) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_fc_input, dim3(rows), dim3(256), 0, st, h, hf, h_row, E, next_tok,
                     visual, d, out);
}

size_t topk_scratch_floats(int rows, int V) {
  const int n_slices = (V + TOPK_SLICE - 1) / TOPK_SLICE;
  return (size_t)rows * n_slices * (2 * TOPK_MAX + 2);
}

void launch_topk(const float* logits, int rows, int V, int k, int* idx, float* val, float* lse,
                 float* scratch, hipStream_t st) {
  if (rows <= 0) return;
  const int n_slices = (V + TOPK_SLICE - 1) / TOPK_SLICE;
  float* cand_v = scratch;
  int* cand_i = reinterpret_cast<int*>(cand_v + (size_t)rows * n_slices * TOPK_MAX);
  float2* stats = reinterpret_cast<float2*>(cand_i + (size_t)rows * n_slices * TOPK_MAX);
  hipLaunchKernelGGL(k_topk_slice, dim3(rows * n_slices), dim3(256), 0, st, logits, V, k, n_slices,
                     cand_v, cand_i, stats);
  hipLaunchKernelGGL(k_topk_merge, dim3(rows), dim3(256), 0, st, k, n_slices, cand_v, cand_i,
                     stats, idx, val, lse);
}

}  // namespace msd
