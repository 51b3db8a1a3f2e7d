// Row-wise kernels of the decode path: embedding gather, RMSNorm, rotary
// embedding with the KV-cache write, the draft input builder and the
// vocabulary top-k / logsumexp.
#include <algorithm>

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
  // 8-element units, every load issued before the first store (d <= 8192)
  uint4 bits[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int u = threadIdx.x + 256 * k;
    bits[k] = 8 * u < d ? *reinterpret_cast<const uint4*>(src + 8 * u) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int u = threadIdx.x + 256 * k;
    if (8 * u >= d) continue;
    const uint32_t w[4] = {bits[k].x, bits[k].y, bits[k].z, bits[k].w};
    float4* o = reinterpret_cast<float4*>(dst + 8 * u);
    o[0] = make_float4(bf2f(w[0] & 0xFFFF), bf2f(w[0] >> 16), bf2f(w[1] & 0xFFFF), bf2f(w[1] >> 16));
    o[1] = make_float4(bf2f(w[2] & 0xFFFF), bf2f(w[2] >> 16), bf2f(w[3] & 0xFFFF), bf2f(w[3] >> 16));
  }
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

// Overwrites the visual rows of x with the target's features of those rows
// (h: split rows of d): the draft input of the Visual Feature variant.
__global__ __launch_bounds__(256) void k_visual_feature_rows(const uint16_t* h, const int* vis_idx,
                                                             int d, float* x) {
  const int row = blockIdx.x;
  if (vis_idx[row] < 0) return;
  const uint16_t* hr = h + (size_t)row * 2 * d;
  for (int e = threadIdx.x; e < d; e += 256) x[(size_t)row * d + e] = get_split(hr, d, e);
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

// Sum over the K chunks of one partial-product element, in chunk order.
// The chunks are loaded in groups of PG, all loads of a group in flight at
// once (indices past the last chunk reload the last one and are not added):
// a loop over a runtime count would otherwise wait for each load of its
// remainder before issuing the next.  The launchers take PG = the chunk
// count rounded up to a power of two, at most MAX_PART_GROUP, so that most
// sums wait for memory once and few loads are repeats.  PART_GROUP: the
// group of the per-row sums of squares (at most eight blocks).
constexpr int PART_GROUP = 8;
constexpr int MAX_PART_GROUP = 16;
inline int part_group(int S) { return S <= 2 ? 2 : S <= 4 ? 4 : S <= 8 ? 8 : MAX_PART_GROUP; }

// Sums over the K chunks of N elements of one row (N columns; every load of a
// chunk group, for all N, in flight at once), in chunk order per element.
// The first group is outside the loop: at a loop head the compiler waits for
// every load in flight, including the caller's.  Entries past the last chunk
// are masked to +0 bitwise rather than skipped: a branch per entry would also
// make the compiler wait at each branch.
MSD_DEV float keep_if(float v, uint32_t m) { return __uint_as_float(__float_as_uint(v) & m); }
template <int N, int PG>
MSD_DEV void part_sums_group(const Parts& pt, const float* p, int s0, const int (&col)[N],
                             float (&out)[N]) {
  float q[N][PG];
#pragma unroll
  for (int n = 0; n < N; ++n)
#pragma unroll
    for (int j = 0; j < PG; ++j)
      q[n][j] = p[col[n] + (size_t)min(s0 + j, pt.S - 1) * pt.split];
#pragma unroll
  for (int j = 0; j < PG; ++j) {
    const uint32_t m = s0 + j < pt.S ? 0xFFFFFFFFu : 0u;
#pragma unroll
    for (int n = 0; n < N; ++n) out[n] += keep_if(q[n][j], m);
  }
}

template <int N, int PG>
MSD_DEV void part_sums(const Parts& pt, int row, const int (&col)[N], float (&out)[N]) {
  const float* p = pt.p + (size_t)row * pt.ld;
#pragma unroll
  for (int n = 0; n < N; ++n) out[n] = 0.f;
  part_sums_group<N, PG>(pt, p, 0, col, out);
  for (int s0 = PG; s0 < pt.S; s0 += PG) part_sums_group<N, PG>(pt, p, s0, col, out);
}

template <int N, int PG>
MSD_DEV void part_sums4_group(const Parts& pt, const float* p, int s0, const int (&col)[N],
                              float4 (&out)[N]) {
  float4 q[N][PG];
#pragma unroll
  for (int n = 0; n < N; ++n)
#pragma unroll
    for (int j = 0; j < PG; ++j)
      q[n][j] = *reinterpret_cast<const float4*>(p + col[n] +
                                                 (size_t)min(s0 + j, pt.S - 1) * pt.split);
#pragma unroll
  for (int j = 0; j < PG; ++j) {
    const uint32_t m = s0 + j < pt.S ? 0xFFFFFFFFu : 0u;
#pragma unroll
    for (int n = 0; n < N; ++n)
      out[n] = make_float4(out[n].x + keep_if(q[n][j].x, m), out[n].y + keep_if(q[n][j].y, m),
                           out[n].z + keep_if(q[n][j].z, m), out[n].w + keep_if(q[n][j].w, m));
  }
}

template <int N, int PG>
MSD_DEV void part_sums4(const Parts& pt, int row, const int (&col)[N], float4 (&out)[N]) {
  const float* p = pt.p + (size_t)row * pt.ld;
#pragma unroll
  for (int n = 0; n < N; ++n) out[n] = make_float4(0.f, 0.f, 0.f, 0.f);
  part_sums4_group<N, PG>(pt, p, 0, col, out);
  for (int s0 = PG; s0 < pt.S; s0 += PG) part_sums4_group<N, PG>(pt, p, s0, col, out);
}

// The same for four consecutive elements (col a multiple of 4).
template <int PG>
MSD_DEV float4 part_sum4(const Parts& pt, int row, int col) {
  const int c[1] = {col};
  float4 o[1];
  part_sums4<1, PG>(pt, row, c, o);
  return o[0];
}

// Four consecutive values of a split row (hi halves at row[k..], lo halves
// at row[K + k..]; k a multiple of 4).
MSD_DEV void put_split4(uint16_t* row, int K, int k, const float (&v)[4]) {
  uint16_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    h[e] = f2bf(v[e]);
    l[e] = f2bf(v[e] - bf2f(h[e]));
  }
  *reinterpret_cast<uint2*>(row + k) =
      make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
  *reinterpret_cast<uint2*>(row + K + k) =
      make_uint2(l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16));
}

// 1 / sqrt(mean(x^2) + eps) of a row from its per-block sums of squares
// (summed in block order); 1 when no sums are given.  ssq_begin issues the
// loads of the first PART_GROUP sums, so that the caller can issue its own
// loads before ssq_end waits for them.
MSD_DEV void ssq_begin(const RowNorm& rn, int row, float (&v)[PART_GROUP]) {
  if (!rn.ssq) return;
  const float* p = rn.ssq + (size_t)row * rn.nblk;
#pragma unroll
  for (int j = 0; j < PART_GROUP; ++j) v[j] = p[min(j, rn.nblk - 1)];
}

MSD_DEV float ssq_end(const RowNorm& rn, int row, const float (&v)[PART_GROUP]) {
  if (!rn.ssq) return 1.f;
  float t = 0.f;
#pragma unroll
  for (int j = 0; j < PART_GROUP; ++j) t += keep_if(v[j], j < rn.nblk ? 0xFFFFFFFFu : 0u);
  const float* p = rn.ssq + (size_t)row * rn.nblk;
  for (int q = PART_GROUP; q < rn.nblk; ++q) t += p[q];
  return rsqrtf(t / (float)rn.d + rn.eps);
}

MSD_DEV float row_rstd(const RowNorm& rn, int row) {
  float v[PART_GROUP];
  ssq_begin(rn, row, v);
  return ssq_end(rn, row, v);
}

// Rotate-half RoPE on q and k, write q (split rows), K to its slot and V to
// the transposed V cache (bf16).  qkv: summed parts, [rows][(H + 2KV) * hd], computed
// from the un-normalised input, so every row is first scaled by its 1/rms.
// Heads H.. are the key heads, H+KV.. the value heads.  One thread per
// (row, head, rotation pair i): a block of ROPE_THREADS threads covers
// ROPE_THREADS / (hd/2) heads of one row (hd/2 divides ROPE_THREADS).
constexpr int ROPE_THREADS = 256;
template <int PG>
__global__ __launch_bounds__(ROPE_THREADS) void k_rope_kv(Parts qkv, RowNorm rn, int H, int KV,
                                                          int hd, const int* pos,
                                                          const int* row_seq,
                                                          const int* row_slot, const float2* tab,
                                                          uint16_t* q, uint16_t* kc,
                                                          uint16_t* vc, int S) {
  const int row = blockIdx.x;
  const int half = hd / 2;
  const int head = blockIdx.y * (ROPE_THREADS / half) + threadIdx.x / half;
  const int i = threadIdx.x % half;
  const int slot = row_slot[row];
  const int b = row_seq[row];
  if (head >= H + 2 * KV || (head >= H && slot < 0)) return;
  // every load (sums of squares, table row, partials) issued before the
  // first use
  float sq[PART_GROUP];
  ssq_begin(rn, row, sq);
  const float2 t = tab[(size_t)pos[row] * half + i];
  const int cols[2] = {head * hd + i, head * hd + i + half};
  float ac[2];
  part_sums<2, PG>(qkv, row, cols, ac);
  const float r = ssq_end(rn, row, sq);
  const float a = r * ac[0];
  const float c = r * ac[1];
  if (head >= H + KV) {
    const int g = head - H - KV;
    uint16_t* vr = vc + (size_t)(b * KV + g) * hd * S + slot;
    vr[(size_t)i * S] = f2bf(a);
    vr[(size_t)(i + half) * S] = f2bf(c);
    return;
  }
  const float y0 = a * t.x - c * t.y;
  const float y1 = c * t.x + a * t.y;
  if (head < H) {
    uint16_t* qr = q + (size_t)row * 2 * H * hd;
    put_split(qr, H * hd, head * hd + i, y0);
    put_split(qr, H * hd, head * hd + i + half, y1);
  } else {
    uint16_t* kr = kc + ((size_t)(b * KV + head - H) * S + slot) * hd;
    kr[i] = f2bf(y0);
    kr[i + half] = f2bf(y1);
  }
}

MSD_DEV float block_sum_1024(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int q = 0; q < 16; ++q) t += sh[q];
  return t;
}

// x = sum of parts (RN_SET), x + sum (RN_ADD) or x (RN_KEEP); then the
// RMSNorm of the new x (gain g) and/or a copy of x, as split rows.  One
// block of 1024 threads per row.
template <int PG>
__global__ __launch_bounds__(1024) void k_resid_norm(Parts pt, int col0, int d, int mode, float* x,
                                                     const uint16_t* g, float eps, uint16_t* xn,
                                                     uint16_t* xb) {
  __shared__ float sh[16];
  const int row = blockIdx.x;
  float* xr = x + (size_t)row * d;
  // four consecutive features per thread and unit, at most two units per
  // thread (d <= 8192); loads issued before their first use, values kept in
  // registers for the normalisation
  constexpr int U = 2;
  float4 v[U], p[U];
  int cols[U];
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int e = 4 * (threadIdx.x + 1024 * k);
    cols[k] = col0 + min(e, d - 4);
    v[k] = e < d ? *reinterpret_cast<const float4*>(xr + e) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  if (mode != RN_KEEP) part_sums4<U, PG>(pt, row, cols, p);
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int e = 4 * (threadIdx.x + 1024 * k);
    if (e >= d) continue;
    if (mode != RN_KEEP) {
      v[k] = (mode == RN_SET) ? p[k]
                              : make_float4(v[k].x + p[k].x, v[k].y + p[k].y, v[k].z + p[k].z,
                                            v[k].w + p[k].w);
      *reinterpret_cast<float4*>(xr + e) = v[k];
    }
    ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
    const float vals[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
    if (xb) put_split4(xb + (size_t)row * 2 * d, d, e, vals);
  }
  if (!g) return;
  ss = block_sum_1024(ss, sh);
  const float r = rsqrtf(ss / (float)d + eps);
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int e = 4 * (threadIdx.x + 1024 * k);
    if (e >= d) continue;
    const uint2 gg = *reinterpret_cast<const uint2*>(g + e);
    const float o[4] = {v[k].x * r * bf2f(gg.x & 0xFFFF), v[k].y * r * bf2f(gg.x >> 16),
                        v[k].z * r * bf2f(gg.y & 0xFFFF), v[k].w * r * bf2f(gg.y >> 16)};
    put_split4(xn + (size_t)row * 2 * d, d, e, o);
  }
}

// Elementwise residual update: x = sum of parts (RN_SET), x + sum (RN_ADD)
// or x (RN_KEEP); then xg = x * g (the next GEMM's input, normalised later
// by its consumer) and xb = x as split rows, and the block's sum of x^2 into
// ssq[row][block].  Grid (ceil(d/256), rows).
// Four consecutive features per thread; a block covers SSQ_BLOCK features of
// one row and writes their sum of squares.  d is a multiple of 4.
template <int PG>
__global__ __launch_bounds__(256) void k_resid(Parts pt, int d, int mode, float* x,
                                               const uint16_t* g, uint16_t* xg, uint16_t* xb,
                                               float* ssq, const int* dst, float* feat) {
  __shared__ float sh[4];
  const int row = blockIdx.y;
  const int e = blockIdx.x * SSQ_BLOCK + 4 * threadIdx.x;
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (e < d) {
    float* const xr = x + (size_t)row * d + e;
    float4 x4 = *reinterpret_cast<const float4*>(xr);
    if (mode != RN_KEEP) {
      const float4 p = part_sum4<PG>(pt, row, e);
      x4 = (mode == RN_SET) ? p : make_float4(x4.x + p.x, x4.y + p.y, x4.z + p.z, x4.w + p.w);
      *reinterpret_cast<float4*>(xr) = x4;
    }
    v[0] = x4.x;
    v[1] = x4.y;
    v[2] = x4.z;
    v[3] = x4.w;
    if (feat) {
      const int o = dst[row];
      if (o >= 0) *reinterpret_cast<float4*>(feat + (size_t)o * d + e) = x4;
    }
    if (xg) {
      const uint2 gb = *reinterpret_cast<const uint2*>(g + e);
      const float vg[4] = {v[0] * bf2f(gb.x & 0xFFFF), v[1] * bf2f(gb.x >> 16),
                           v[2] * bf2f(gb.y & 0xFFFF), v[3] * bf2f(gb.y >> 16)};
      put_split4(xg + (size_t)row * 2 * d, d, e, vg);
    }
    if (xb) put_split4(xb + (size_t)row * 2 * d, d, e, v);
  }
  if (!ssq) return;
  const float t = block_sum_256(v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3], sh);
  if (threadIdx.x == 0) ssq[(size_t)row * gridDim.x + blockIdx.x] = t;
}

// x[i] = the last feature of sequence seq_ids[i] (its feature slot 0), xb
// the same as a split row; four features per thread.
__global__ __launch_bounds__(256) void k_root_feat(const int* seq_ids, const float* feat,
                                                   int feat_stride, int d, float* x,
                                                   uint16_t* xb) {
  const int i = blockIdx.y;
  const int e = blockIdx.x * 1024 + 4 * threadIdx.x;
  if (e >= d) return;
  const float4 v =
      *reinterpret_cast<const float4*>(feat + (size_t)seq_ids[i] * feat_stride * d + e);
  *reinterpret_cast<float4*>(x + (size_t)i * d + e) = v;
  const float w[4] = {v.x, v.y, v.z, v.w};
  put_split4(xb + (size_t)i * 2 * d, d, e, w);
}

// act = silu(gate) * up (split rows) with gate at columns [0, F), up at
// [off2, off2 + F), both scaled by the row's 1/rms (the GEMM read the
// un-normalised input).
template <int PG>
__global__ __launch_bounds__(256) void k_silu(Parts pt, RowNorm rn, int F, uint16_t* act) {
  const int row = blockIdx.y;
  const int f = blockIdx.x * 1024 + 4 * threadIdx.x;  // F is a multiple of 4
  if (f >= F) return;
  float sq[PART_GROUP];
  ssq_begin(rn, row, sq);
  const int cols[2] = {f, pt.off2 + f};
  float4 gu[2];
  part_sums4<2, PG>(pt, row, cols, gu);
  const float r = ssq_end(rn, row, sq);
  const float4 gt = gu[0], up = gu[1];
  const float g4[4] = {gt.x, gt.y, gt.z, gt.w}, u4[4] = {up.x, up.y, up.z, up.w};
  float o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float gv = r * g4[e];
    o[e] = gv / (1.f + __expf(-gv)) * (r * u4[e]);
  }
  put_split4(act + (size_t)row * 2 * F, F, f, o);
}

// out[row] = [h_row | e_next] as a split row of 2d, the concat fed to the
// draft's f_down; h rows are target features (split rows, h) or draft
// features (float32 rows, hf); next_tok >= 0 selects E[next_tok], next_tok < 0
// selects visual row -1-next_tok.  Grid (rows, ceil(d/256)).
__global__ __launch_bounds__(256) void k_fc_input(const uint16_t* h, const float* hf,
                                                  const int* h_row, const uint16_t* E,
                                                  const int* next_tok, const uint16_t* visual,
                                                  int d, uint16_t* out) {
  const int row = blockIdx.x;
  const int hr = h_row[row];
  const int nt = next_tok[row];
  const uint16_t* e = (nt >= 0) ? E + (size_t)nt * d : visual + (size_t)(-1 - nt) * d;
  uint16_t* o = out + (size_t)row * 4 * d;
  const int i = blockIdx.y * 256 + threadIdx.x;
  if (i < d) {
    if (h) {
      const uint16_t* hs = h + (size_t)hr * 2 * d;
      o[i] = hs[i];
      o[2 * d + i] = hs[d + i];
    } else {
      put_split(o, 2 * d, i, hf[(size_t)hr * d + i]);
    }
    o[d + i] = e[i];
    o[3 * d + i] = 0;
  }
}

// Per-row top-k over the vocabulary (value descending, then id ascending)
// and the row's logsumexp, in two phases: every (row, slice) block reduces a
// slice of the vocabulary to its own top-k and (max, sum of exp) pair; one
// block per row then merges the slices (logsumexp in slice order).  The
// order is total, so the result does not depend on how candidates are
// partitioned.
constexpr int TOPK_MAX = 16;
constexpr int TOPK_SLICE = 2048;

MSD_DEV bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

constexpr int TOPK_PER = TOPK_SLICE / 256;  // logits per thread of a slice block
constexpr int TOPK_MERGE_PER = 8;           // slice candidates per thread of the merge
constexpr int NO_ID = 0x7FFFFFFF;           // an absent candidate (ranks after every id)

// The wave's best (value, id) over its lanes' offers.
MSD_DEV void wave_best(float& v, int& id) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(v, o);
    const int oi = __shfl_xor(id, o);
    if (better(ov, oi, v, id)) {
      v = ov;
      id = oi;
    }
  }
}

// The k best of the wave's candidates (N per lane, ids unique apart from
// NO_ID), best first: k rounds of a wave-wide argmax in which the owner of
// the winner retires it.  Lane 0 writes them to out_v / out_i.
template <int N>
MSD_DEV void wave_select(const float (&cv)[N], const int (&ci)[N], int k, float* out_v,
                         int* out_i) {
  uint32_t taken = 0;
  for (int q = 0; q < k; ++q) {
    float bv = -INFINITY;
    int bi = NO_ID, bj = -1;
#pragma unroll
    for (int j = 0; j < N; ++j) {
      if (!((taken >> j) & 1u) && better(cv[j], ci[j], bv, bi)) {
        bv = cv[j];
        bi = ci[j];
        bj = j;
      }
    }
    float wv = bv;
    int wi = bi;
    wave_best(wv, wi);
    if (bj >= 0 && bi == wi) taken |= 1u << bj;
    if ((threadIdx.x & 63) == 0) {
      out_v[q] = wv;
      out_i[q] = wi;
    }
  }
}

// The k best of the 4 waves' lists (wv/wi[w][0..k)), selected by wave 0.
MSD_DEV void block_merge(const float (*wv)[TOPK_MAX], const int (*wi)[TOPK_MAX], int k,
                         float* out_v, int* out_i) {
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  float c[1] = {lane < 4 * k ? wv[lane / k][lane % k] : -INFINITY};
  int ci[1] = {lane < 4 * k ? wi[lane / k][lane % k] : NO_ID};
  wave_select<1>(c, ci, k, out_v, out_i);
}

template <int PG>
__global__ __launch_bounds__(256) void k_topk_slice(Parts logits, int V, int k, int n_slices,
                                                    float* cand_v, int* cand_i, float2* stats,
                                                    float* logits_out) {
  __shared__ float wv[4][TOPK_MAX];
  __shared__ int wi[4][TOPK_MAX];
  __shared__ float sm[4];
  __shared__ float ssum[4];
  const int row = blockIdx.x / n_slices;
  const int sl = blockIdx.x - row * n_slices;
  const int v0 = sl * TOPK_SLICE;
  float cv[TOPK_PER];
  int ci[TOPK_PER];
  float mloc = -INFINITY, sloc = 0.f;
  int cols[TOPK_PER];
#pragma unroll
  for (int e = 0; e < TOPK_PER; ++e) cols[e] = min(v0 + threadIdx.x + 256 * e, V - 1);
  float raws[TOPK_PER];
  part_sums<TOPK_PER, PG>(logits, row, cols, raws);
#pragma unroll
  for (int e = 0; e < TOPK_PER; ++e) {
    const int v = v0 + threadIdx.x + 256 * e;
    float val = -INFINITY;
    int id = NO_ID;
    if (v < V) {
      const float raw = raws[e];
      if (logits_out) logits_out[(size_t)row * V + v] = raw;
      // a NaN ranks as -inf, so the selected ids are always vocabulary ids
      val = (raw == raw) ? raw : -INFINITY;
      id = v;
      if (val > mloc) {
        sloc = sloc * __expf(mloc - val) + 1.f;
        mloc = val;
      } else if (val != -INFINITY) {
        sloc += __expf(val - mloc);
      }
    }
    cv[e] = val;
    ci[e] = id;
  }
  float mm = mloc;
  for (int o = 32; o > 0; o >>= 1) mm = fmaxf(mm, __shfl_xor(mm, o));
  if ((threadIdx.x & 63) == 0) sm[threadIdx.x >> 6] = mm;
  __syncthreads();
  const float M = fmaxf(fmaxf(sm[0], sm[1]), fmaxf(sm[2], sm[3]));
  const float part = (mloc == -INFINITY) ? 0.f : sloc * __expf(mloc - M);
  const float tot = block_sum_256(part, ssum);
  if (threadIdx.x == 0) stats[blockIdx.x] = make_float2(M, tot);
  const int w = threadIdx.x >> 6;
  wave_select<TOPK_PER>(cv, ci, k, wv[w], wi[w]);
  __syncthreads();
  block_merge(wv, wi, k, cand_v + (size_t)blockIdx.x * k, cand_i + (size_t)blockIdx.x * k);
}

// (m, t) <- the merge of two (max, sum of exp(x - max)) pairs.
MSD_DEV void lse_merge(float& m, float& t, float m2, float t2) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) {
    m = m2;
    t = t2;
  } else if (m2 > m) {
    t = t * __expf(m - m2) + t2;
    m = m2;
  } else {
    t += t2 * __expf(m2 - m);
  }
}

// One block per row merges its slices' candidates (n_slices * k of them,
// at most 256 * TOPK_MERGE_PER) and their logsumexp parts.
__global__ __launch_bounds__(256) void k_topk_merge(int k, int n_slices, const float* cand_v,
                                                    const int* cand_i, const float2* stats,
                                                    int* out_idx, float* out_val, float* out_lse) {
  __shared__ float wv[4][TOPK_MAX];
  __shared__ int wi[4][TOPK_MAX];
  __shared__ float fv[TOPK_MAX];
  __shared__ int fi[TOPK_MAX];
  const int row = blockIdx.x;
  const int n = n_slices * k;
  const size_t c0 = (size_t)row * n;
  float cv[TOPK_MERGE_PER];
  int ci[TOPK_MERGE_PER];
#pragma unroll
  for (int e = 0; e < TOPK_MERGE_PER; ++e) {
    const int c = threadIdx.x + 256 * e;
    cv[e] = c < n ? cand_v[c0 + c] : -INFINITY;
    ci[e] = c < n ? cand_i[c0 + c] : NO_ID;
  }
  const int w = threadIdx.x >> 6;
  wave_select<TOPK_MERGE_PER>(cv, ci, k, wv[w], wi[w]);
  __syncthreads();
  block_merge(wv, wi, k, fv, fi);
  __syncthreads();
  if (threadIdx.x < k) {
    out_idx[(size_t)row * k + threadIdx.x] = fi[threadIdx.x];
    if (out_val) out_val[(size_t)row * k + threadIdx.x] = fv[threadIdx.x];
  }
  if (out_lse) {
    // logsumexp over the slices' (max, sum of exp) pairs: every thread merges
    // its slices, then the waves and the block merge in a fixed order
    const float2* st = stats + (size_t)row * n_slices;
    float m = -INFINITY, t = 0.f;
    for (int q = threadIdx.x; q < n_slices; q += 256) lse_merge(m, t, st[q].x, st[q].y);
    for (int o = 32; o > 0; o >>= 1) lse_merge(m, t, __shfl_xor(m, o), __shfl_xor(t, o));
    __shared__ float lm[4], lt[4];
    if ((threadIdx.x & 63) == 0) {
      lm[threadIdx.x >> 6] = m;
      lt[threadIdx.x >> 6] = t;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      float M = -INFINITY, T = 0.f;
      for (int w = 0; w < 4; ++w) lse_merge(M, T, lm[w], lt[w]);
      out_lse[row] = M + __logf(T);
    }
  }
}

}  // namespace

// Launches kernel template K<PG> with PG = part_group(S).
#define PG_DISPATCH(S, K, ...)                                       \
  do {                                                               \
    switch (part_group(S)) {                                         \
      case 2: hipLaunchKernelGGL(K<2>, __VA_ARGS__); break;          \
      case 4: hipLaunchKernelGGL(K<4>, __VA_ARGS__); break;          \
      case 8: hipLaunchKernelGGL(K<8>, __VA_ARGS__); break;          \
      default: hipLaunchKernelGGL(K<MAX_PART_GROUP>, __VA_ARGS__);   \
    }                                                                \
  } while (0)

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

void launch_visual_feature_rows(const uint16_t* h, const int* vis_idx, int rows, int d, float* x,
                                hipStream_t st) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_visual_feature_rows, dim3(rows), dim3(256), 0, st, h, vis_idx, d, x);
}

void launch_rope_table(float2* tab, int max_pos, int hd, double theta, hipStream_t st) {
  const int n = max_pos * (hd / 2);
  hipLaunchKernelGGL(k_rope_table, dim3((n + 255) / 256), dim3(256), 0, st, tab, max_pos,
                     hd / 2, theta);
}

void launch_rope_kv(Parts qkv, RowNorm rn, int rows, int H, int KV, int hd, const int* pos,
                    const int* row_seq, const int* row_slot, const float2* rope_tab,
                    uint16_t* q, uint16_t* kc, uint16_t* vc, int S, hipStream_t st) {
  if (rows <= 0) return;
  const int per_block = ROPE_THREADS / (hd / 2);
  const dim3 grid(rows, (H + 2 * KV + per_block - 1) / per_block);
  PG_DISPATCH(qkv.S, k_rope_kv, grid, dim3(ROPE_THREADS), 0, st, qkv, rn, H, KV, hd, pos, row_seq,
              row_slot, rope_tab, q, kc, vc, S);
}

void launch_resid_norm(Parts pt, int col0, int rows, int d, int mode, float* x,
                       const uint16_t* g, float eps, uint16_t* xn, uint16_t* xb, hipStream_t st) {
  if (rows <= 0) return;
  // groups of at most 8: at 16 the 1024-thread blocks' registers spill
  const int pg = part_group(std::min(pt.S, 8));
  if (pg == 2)
    hipLaunchKernelGGL(k_resid_norm<2>, dim3(rows), dim3(1024), 0, st, pt, col0, d, mode, x, g,
                       eps, xn, xb);
  else if (pg == 4)
    hipLaunchKernelGGL(k_resid_norm<4>, dim3(rows), dim3(1024), 0, st, pt, col0, d, mode, x, g,
                       eps, xn, xb);
  else
    hipLaunchKernelGGL(k_resid_norm<8>, dim3(rows), dim3(1024), 0, st, pt, col0, d, mode, x, g,
                       eps, xn, xb);
}

void launch_root_feat(int n_seq, const int* seq_ids, const float* feat, int feat_stride, int d,
                      float* x, uint16_t* xb, hipStream_t st) {
  if (n_seq <= 0) return;
  hipLaunchKernelGGL(k_root_feat, dim3((d + 1023) / 1024, n_seq), dim3(256), 0, st, seq_ids,
                     feat, feat_stride, d, x, xb);
}

void launch_silu(Parts pt, RowNorm rn, int rows, int F, uint16_t* act, hipStream_t st) {
  if (rows <= 0) return;
  PG_DISPATCH(pt.S, k_silu, dim3((F + 1023) / 1024, rows), dim3(256), 0, st, pt, rn, F, act);
}

void launch_resid(Parts pt, int rows, int d, int mode, float* x, const uint16_t* g, uint16_t* xg,
                  uint16_t* xb, float* ssq, hipStream_t st, const int* dst, float* feat) {
  if (rows <= 0) return;
  PG_DISPATCH(pt.S, k_resid, dim3(ssq_blocks(d), rows), dim3(256), 0, st, pt, d, mode, x, g, xg,
              xb, ssq, dst, feat);
}

void launch_fc_input(const uint16_t* h, const float* hf, const int* h_row, const uint16_t* E,
                     const int* next_tok, const uint16_t* visual, int rows, int d, uint16_t* out,
                     hipStream_t st) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_fc_input, dim3(rows, (d + 255) / 256), dim3(256), 0, st, h, hf, h_row, E,
                     next_tok, visual, d, out);
}

size_t topk_scratch_floats(int rows, int V) {
  const int n_slices = (V + TOPK_SLICE - 1) / TOPK_SLICE;
  return (size_t)rows * n_slices * (2 * TOPK_MAX + 2);
}

void launch_topk(Parts logits, int rows, int V, int k, int* idx, float* val, float* lse,
                 float* logits_out, float* scratch, hipStream_t st) {
  if (rows <= 0) return;
  const int n_slices = (V + TOPK_SLICE - 1) / TOPK_SLICE;
  float* cand_v = scratch;
  int* cand_i = reinterpret_cast<int*>(cand_v + (size_t)rows * n_slices * TOPK_MAX);
  float2* stats = reinterpret_cast<float2*>(cand_i + (size_t)rows * n_slices * TOPK_MAX);
  PG_DISPATCH(logits.S, k_topk_slice, dim3(rows * n_slices), dim3(256), 0, st, logits, V, k,
              n_slices, cand_v, cand_i, stats, logits_out);
  hipLaunchKernelGGL(k_topk_merge, dim3(rows), dim3(256), 0, st, k, n_slices, cand_v, cand_i,
                     stats, idx, val, lse);
}

}  // namespace msd
