// Speculative sampling on a verified tree at temperature > 0 (Sec. 3.2,
// verification phase: acceptance probability min(1, p/q) and the adjusted
// distribution norm(max(0, p - q)) after a rejection).
//
// The drafted children of a node are the draft's top-ranked tokens, a
// deterministic choice, so each child's proposal is the point mass on its
// token: a child is accepted with probability p(x) / (1 - mass already
// rejected at this node), a rejection removes x from p, and when no child is
// accepted the bonus token is drawn from p without the rejected tokens.  An
// accepted child's own children are tried next against the target
// distribution at that child.  p = softmax(logits / temperature) per node.
//
// One 1024-thread block per sequence.  Every thread takes the same decisions
// (block-wide reductions end in the same fixed-order merge on every thread);
// thread 0 records the path and the rejected tokens in LDS.
//
// Uniforms: draw j of the cycle of sequence slot b starting at committed
// length L is output n = b * 2^40 + L * 2^8 + j of SplitMix64 (Steele, Lea and
// Flood, 2014) started at the caller's seed; its top 24 bits scaled by 2^-24.
#include <math.h>

#include "../../include/msd.h"
#include "msd_internal.h"

namespace msd {

namespace {

constexpr int SAMPLE_THREADS = 1024;
constexpr int SAMPLE_WAVES = SAMPLE_THREADS / 64;

MSD_DEV uint64_t splitmix64(uint64_t seed, uint64_t n) {
  uint64_t z = seed + (n + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

MSD_DEV float draw_uniform(uint64_t seed, int b, int L, int j) {
  const uint64_t n = ((uint64_t)b << 40) | ((uint64_t)(uint32_t)L << 8) | (uint64_t)j;
  return (float)(uint32_t)(splitmix64(seed, n) >> 40) * 0x1p-24f;
}

// Scaled logit; NaN ranks as -inf (zero probability).
MSD_DEV float scaled(const float* lg, int v, float inv_t) {
  const float z = lg[v] * inv_t;
  return z == z ? z : -INFINITY;
}

// (m, s) <- merge with (m2, s2), where s sums exp(z - m).
MSD_DEV void ms_merge(float& m, float& s, float m2, float s2) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) {
    m = m2;
    s = s2;
  } else if (m2 > m) {
    s = s * expf(m - m2) + s2;
    m = m2;
  } else {
    s += s2 * expf(m2 - m);
  }
}

// Max and sum of exp(z - max) over the row; identical on every thread.
MSD_DEV void row_stats(const float* lg, int V, float inv_t, float* sh_m, float* sh_s, float& m,
                       float& s) {
  m = -INFINITY;
  s = 0.f;
  for (int v = threadIdx.x; v < V; v += SAMPLE_THREADS) ms_merge(m, s, scaled(lg, v, inv_t), 1.f);
  for (int o = 32; o > 0; o >>= 1) ms_merge(m, s, __shfl_xor(m, o), __shfl_xor(s, o));
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    sh_m[w] = m;
    sh_s[w] = s;
  }
  __syncthreads();
  m = -INFINITY;
  s = 0.f;
  for (int i = 0; i < SAMPLE_WAVES; ++i) ms_merge(m, s, sh_m[i], sh_s[i]);
}

MSD_DEV bool is_rejected(int v, const int* rej, int n_rej) {
  for (int i = 0; i < n_rej; ++i)
    if (rej[i] == v) return true;
  return false;
}

__global__ __launch_bounds__(SAMPLE_THREADS) void k_accept_sample(
    const msd_tree* trees, const int* seq_ids, int T, const float* logits, int V, float inv_t,
    uint64_t seed, int* path, int* n_path, int* emitted, int* slot_map, const int* d_len,
    const int* tree_err, int n_seq) {
  __shared__ float sh_m[SAMPLE_WAVES], sh_s[SAMPLE_WAVES], sh_w[SAMPLE_WAVES];
  __shared__ int sh_path[MSD_MAX_TREE], sh_rej[MSD_MAX_TREE];
  __shared__ int sh_y;
  __shared__ float sh_bv[SAMPLE_WAVES];
  __shared__ int sh_bi[SAMPLE_WAVES];
  const int sidx = blockIdx.x;
  const msd_tree* t = trees + sidx;
  const int b = seq_ids[sidx];
  const int L = d_len[b];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (any_tree_err(tree_err, n_seq)) {  // a flagged call accepts nothing
    for (int j = threadIdx.x; j < MSD_MAX_TREE; j += SAMPLE_THREADS) {
      path[sidx * MSD_MAX_TREE + j] = -1;
      slot_map[sidx * MSD_MAX_TREE + j] = -1;
      emitted[sidx * MSD_MAX_TREE + j] = -1;
    }
    if (threadIdx.x == 0) n_path[sidx] = 0;
    return;
  }
  if (threadIdx.x == 0) sh_path[0] = 0;
  int cur = 0, n = 1, jd = 0, n_rej = 0;
  const float* lg = logits;
  float m = 0.f, s = 0.f;
  for (;;) {
    lg = logits + ((size_t)sidx * T + cur) * V;
    row_stats(lg, V, inv_t, sh_m, sh_s, m, s);
    float removed = 0.f;
    int next = -1;
    n_rej = 0;
    for (int u = cur + 1; u < T; ++u) {
      if (t->parent[u] != cur) continue;
      const int x = min(max(t->token[u], 0), V - 1);
      const float zx = scaled(lg, x, inv_t);
      const float px = zx == -INFINITY ? 0.f : expf(zx - m) / s;
      const float r = draw_uniform(seed, b, L, jd++);
      const float rem = 1.f - removed;  // target mass not yet rejected here
      if (rem > 0.f && r * rem < px) {
        next = u;
        break;
      }
      removed += px;
      if (threadIdx.x == 0) sh_rej[n_rej] = x;
      ++n_rej;
    }
    if (next < 0 || n >= MSD_MAX_TREE) break;
    if (threadIdx.x == 0) sh_path[n] = next;
    ++n;
    cur = next;
  }
  __syncthreads();  // sh_rej, sh_path

  // bonus token: inverse CDF of p without the rejected tokens, each thread
  // owning a contiguous range of the vocabulary
  const float r = draw_uniform(seed, b, L, jd);
  const int cs = (V + SAMPLE_THREADS - 1) / SAMPLE_THREADS;
  const int v0 = min(V, (int)threadIdx.x * cs), v1 = min(V, v0 + cs);
  float part = 0.f;
  for (int v = v0; v < v1; ++v) {
    const float z = scaled(lg, v, inv_t);
    if (z != -INFINITY && !is_rejected(v, sh_rej, n_rej)) part += expf(z - m);
  }
  // inclusive scan in thread order; the intervals [excl, incl) tile [0, total)
  float incl = part;
  for (int o = 1; o < 64; o <<= 1) {
    const float y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) sh_w[w] = incl;
  if (threadIdx.x == 0) sh_y = -1;
  __syncthreads();
  float off = 0.f;
  for (int i = 0; i < w; ++i) off += sh_w[i];
  float total = off;
  for (int i = w; i < SAMPLE_WAVES; ++i) total += sh_w[i];
  const float prev = __shfl_up(incl, 1);
  const float lo = lane == 0 ? off : off + prev;
  const float hi = off + incl;
  const float target = r * total;
  if (total > 0.f && part > 0.f && lo <= target && target < hi) {
    float acc = 0.f;
    int y = -1, last = -1;
    for (int v = v0; v < v1; ++v) {
      const float z = scaled(lg, v, inv_t);
      if (z == -INFINITY || is_rejected(v, sh_rej, n_rej)) continue;
      acc += expf(z - m);
      last = v;
      if (lo + acc > target) {
        y = v;
        break;
      }
    }
    sh_y = y >= 0 ? y : last;
  }
  __syncthreads();
  int y = sh_y;
  if (y < 0) {
    // no mass left in float32: the best remaining logit (lowest id on ties)
    float bv = -INFINITY;
    int bi = V;
    for (int v = v0; v < v1; ++v) {
      const float z = scaled(lg, v, inv_t);
      if (!is_rejected(v, sh_rej, n_rej) && (z > bv || bi == V)) {
        bv = z;
        bi = v;
      }
    }
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o);
      const int oi = __shfl_xor(bi, o);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if (lane == 0) {
      sh_bv[w] = bv;
      sh_bi[w] = bi;
    }
    __syncthreads();
    bv = -INFINITY;
    bi = V;
    for (int i = 0; i < SAMPLE_WAVES; ++i)
      if (sh_bi[i] < V && (sh_bv[i] > bv || bi == V || (sh_bv[i] == bv && sh_bi[i] < bi))) {
        bv = sh_bv[i];
        bi = sh_bi[i];
      }
    y = bi < V ? bi : 0;
  }
  for (int j = threadIdx.x; j < MSD_MAX_TREE; j += SAMPLE_THREADS) {
    const int u = j < n ? sh_path[j] : -1;
    path[sidx * MSD_MAX_TREE + j] = u;
    slot_map[sidx * MSD_MAX_TREE + j] = j < n ? L + u : -1;
    emitted[sidx * MSD_MAX_TREE + j] =
        (j + 1 < n) ? t->token[sh_path[j + 1]] : ((j + 1 == n) ? y : -1);
  }
  if (threadIdx.x == 0) n_path[sidx] = n;
}

}  // namespace

void launch_accept_sample(const void* trees, int n_seq, const int* seq_ids, int T,
                          const float* logits, int V, float inv_t, uint64_t seed, int* path,
                          int* n_path, int* emitted, int* slot_map, const int* d_len,
                          const int* tree_err, hipStream_t st) {
  hipLaunchKernelGGL(k_accept_sample, dim3(n_seq), dim3(SAMPLE_THREADS), 0, st,
                     (const msd_tree*)trees, seq_ids, T, logits, V, inv_t, seed, path, n_path,
                     emitted, slot_map, d_len, tree_err, n_seq);
}

}  // namespace msd
