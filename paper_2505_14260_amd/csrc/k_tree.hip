// Tree bookkeeping kernels: per-step row descriptors, static and dynamic
// draft-tree construction, greedy acceptance and in-place KV compaction.
// All of this is integer / selection work on at most a few hundred entries
// per sequence, so the kernels use one block (or one thread) per sequence.
#include "../../include/msd.h"
#include "msd_internal.h"

namespace msd {

namespace {

MSD_DEV bool better_score(float sa, int ia, float sb, int ib) {
  return sa > sb || (sa == sb && ia < ib);
}

__global__ void k_tree_init_static(msd_tree* trees, const int* seq_ids, const int* d_root,
                                   StaticSpec sp, int T) {
  const int sidx = blockIdx.x;
  msd_tree* t = trees + sidx;
  const int b = seq_ids[sidx];
  for (int i = threadIdx.x; i < MSD_MAX_TREE; i += blockDim.x) {
    const bool in = i < T;
    t->token[i] = (i == 0) ? d_root[b] : 0;
    t->parent[i] = in ? sp.parent[i] : -1;
    t->depth[i] = in ? sp.depth[i] : 0;
    t->anc[i] = in ? sp.anc[i] : 0ull;
    t->score[i] = 0.f;
  }
  if (threadIdx.x == 0) t->n_nodes = T;
}


// Round `depth` (>= 1) of a static tree, one block per (row, 256-feature
// slice).  The row's node takes the rank-th best token of its parent's draft
// distribution (the previous round's top-k, n_prev rows per sequence).  The
// slice-0 block writes the row descriptor; the sequence's first row's slice-0
// block also assigns every node of this depth (leaves included); every block
// gathers its slice of the f_down input [parent feature | token embedding]
// as a split row of 2d.
__global__ __launch_bounds__(256) void k_static_next(msd_tree* trees, const int* seq_ids,
                                                     const int* d_len, StaticSpec sp, int T,
                                                     int depth, const int* topk_idx, int k,
                                                     int n_prev, int round_off, int n_round,
                                                     int feat_stride, Rows r, int* prefix,
                                                     const float* feat, const uint16_t* E, int d,
                                                     uint16_t* out) {
  const int row = blockIdx.x;
  const int sidx = row / n_round, j = row - sidx * n_round;
  const int b = seq_ids[sidx];
  const int u = sp.round_nodes[round_off + j];
  const auto token_of = [&](int c) {
    return topk_idx[(size_t)(sidx * n_prev + sp.round_pos[sp.parent[c]]) * k + sp.rank[c]];
  };
  const int tok = token_of(u);
  if (blockIdx.y == 0) {
    if (threadIdx.x == 0) {
      const int L = d_len[b];
      if (j == 0) prefix[sidx] = L;
      r.tok[row] = tok;
      r.vis[row] = -1;
      r.hrow[row] = b * feat_stride + sp.pslot[u];
      r.pos[row] = L + depth - 1;
      r.slot[row] = L + sp.exp_idx[u];
      r.seq[row] = b;
      r.mask[row] = sp.exp_mask[u];
      r.dst[row] = b * feat_stride + 1 + sp.exp_idx[u];
    }
    if (j == 0)
      for (int c = 1 + threadIdx.x; c < T; c += blockDim.x)
        if (sp.depth[c] == depth) trees[sidx].token[c] = token_of(c);
  }
  const int i = blockIdx.y * 256 + threadIdx.x;
  if (i < d) {
    uint16_t* const o = out + (size_t)row * 4 * d;
    put_split(o, 2 * d, i, feat[(size_t)(b * feat_stride + sp.pslot[u]) * d + i]);
    o[d + i] = E[(size_t)tok * d + i];
    o[3 * d + i] = 0;
  }
}

// Pending draft rows of each sequence, padded to r_max rows per sequence, one
// block per (row, 256-feature slice): the slice-0 block writes the row
// descriptor, every block its slice of the f_down input [pending feature |
// embedding of the next token].  A sequence with no pending row (a padding
// row only) takes token 0 and a zero feature; its row is never stored.
__global__ __launch_bounds__(256) void k_catchup_next(const int* seq_ids, const int* d_len,
                                                      const int* pend_n, const int* pend_next,
                                                      int r_max, int pend_stride, int feat_stride,
                                                      Rows r, int* prefix, const uint16_t* pend_h,
                                                      const uint16_t* E, int d, uint16_t* out) {
  const int row = blockIdx.x;
  const int sidx = row / r_max, j = row - sidx * r_max;
  const int b = seq_ids[sidx];
  const int rb = pend_n[b];
  const bool valid = j < rb;
  const int jj = valid ? j : (rb > 0 ? rb - 1 : 0);
  const int tok = rb > 0 ? pend_next[b * pend_stride + jj] : 0;
  if (blockIdx.y == 0 && threadIdx.x == 0) {
    const int P = d_len[b] - rb;
    if (j == 0) prefix[sidx] = P;
    r.tok[row] = tok;
    r.vis[row] = -1;
    r.hrow[row] = b * pend_stride + jj;
    r.pos[row] = P + jj;
    r.slot[row] = valid ? P + j : -1;
    r.seq[row] = b;
    // causal inside the pending region: row j sees pending rows 0..j
    r.mask[row] = (jj >= 63) ? ~0ull : ((2ull << jj) - 1ull);
    r.dst[row] = (j == rb - 1) ? b * feat_stride : -1;
  }
  const int i = blockIdx.y * 256 + threadIdx.x;
  if (i < d) {
    const uint16_t* const hs = pend_h + (size_t)(b * pend_stride + jj) * 2 * d;
    uint16_t* const o = out + (size_t)row * 4 * d;
    o[i] = rb > 0 ? hs[i] : (uint16_t)0;
    o[2 * d + i] = rb > 0 ? hs[d + i] : (uint16_t)0;
    o[d + i] = E[(size_t)tok * d + i];
    o[3 * d + i] = 0;
  }
}

// Children of the round's nodes: node c with parent p takes the rank[c]-th
// best token of p's draft distribution.
__global__ void k_static_assign(msd_tree* trees, StaticSpec sp, int T, int parent_depth,
                                const int* topk_idx, int k, int n_round) {
  const int sidx = blockIdx.x;
  for (int c = 1 + threadIdx.x; c < T; c += blockDim.x) {
    if (sp.depth[c] != parent_depth + 1) continue;
    const int p = sp.parent[c];
    const int row = sidx * n_round + sp.round_pos[p];
    trees[sidx].token[c] = topk_idx[(size_t)row * k + sp.rank[c]];
  }
}

// Dynamic tree, depth 1: the root's top-K with scores log q.
__global__ void k_dyn_root(DynPool pool, const int* topk_idx, const float* topk_val,
                           const float* lse, int K) {
  const int sidx = blockIdx.x;
  const int j = threadIdx.x;
  if (j >= K) return;
  const size_t o = (size_t)sidx * pool.cap + j;
  pool.parent[o] = -1;
  pool.tok[o] = topk_idx[sidx * K + j];
  pool.depth[o] = 1;
  pool.score[o] = topk_val[sidx * K + j] - lse[sidx];
  pool.exp_idx[o] = j;
  pool.mask[o] = 1ull << j;
  pool.frontier[sidx * K + j] = j;
}

// Rows for expanding the current frontier (nodes of depth depth-1 at draft
// position L + depth - 2).
__global__ void k_dyn_rows(DynPool pool, const int* seq_ids, const int* d_len, int K,
                           int depth, int feat_stride, Rows r, int* prefix) {
  const int sidx = blockIdx.x;
  const int j = threadIdx.x;
  const int b = seq_ids[sidx];
  const int L = d_len[b];
  if (j == 0) prefix[sidx] = L;
  if (j >= K) return;
  const size_t base = (size_t)sidx * pool.cap;
  const int u = pool.frontier[sidx * K + j];
  const int p = pool.parent[base + u];
  const int row = sidx * K + j;
  r.tok[row] = pool.tok[base + u];
  r.vis[row] = -1;
  r.hrow[row] = b * feat_stride + (p < 0 ? 0 : 1 + pool.exp_idx[base + p]);
  r.pos[row] = L + depth - 2;
  r.slot[row] = L + pool.exp_idx[base + u];
  r.seq[row] = b;
  r.mask[row] = pool.mask[base + u];
  r.dst[row] = b * feat_stride + 1 + pool.exp_idx[base + u];
}

// Adds the K*K children of the frontier (frontier order, then rank order),
// picks the best K as the next frontier and gives them expansion indices
// exp_base + position in creation order.
__global__ void k_dyn_expand(DynPool pool, const int* topk_idx, const float* topk_val,
                             const float* lse, int K, int n_pool, int exp_base) {
  __shared__ float sc[256];
  __shared__ int sel[16];
  const int sidx = blockIdx.x;
  const size_t base = (size_t)sidx * pool.cap;
  const int KK = K * K;
  const int t = threadIdx.x;
  if (t < KK) {
    const int j = t / K;
    const int row = sidx * K + j;
    const int u = pool.frontier[sidx * K + j];
    const int id = n_pool + t;
    const float lq = topk_val[(size_t)row * K + (t - j * K)] - lse[row];
    const float s = pool.score[base + u] + lq;
    pool.parent[base + id] = u;
    pool.tok[base + id] = topk_idx[(size_t)row * K + (t - j * K)];
    pool.depth[base + id] = pool.depth[base + u] + 1;
    pool.score[base + id] = s;
    pool.exp_idx[base + id] = -1;
    pool.mask[base + id] = 0ull;
    sc[t] = s;
  }
  __syncthreads();
  if (t < KK) {
    int rank = 0;
    for (int q = 0; q < KK; ++q) rank += better_score(sc[q], q, sc[t], t) ? 1 : 0;
    if (rank < K) sel[rank] = t;
  }
  __syncthreads();
  if (t < K) {
    // position in creation order among the selected
    const int me = sel[t];
    int pos = 0;
    for (int q = 0; q < K; ++q) pos += (sel[q] < me) ? 1 : 0;
    const int id = n_pool + me;
    const int e = exp_base + pos;
    if (e < 64) {  // the last depth's frontier is never expanded
      pool.exp_idx[base + id] = e;
      pool.mask[base + id] = pool.mask[base + pool.parent[base + id]] | (1ull << e);
    }
    pool.frontier[sidx * K + pos] = id;
  }
}

// Final tree: best N of the pool (score desc, creation asc), laid out by
// (depth, creation) with the root as node 0.
// The tree of one sequence from its candidate pool: the N best candidates
// (score descending, then creation order) in canonical order (depth, then
// creation order).  A bitonic sort of the (score, index) keys in LDS puts
// the N best first; the kept candidates are then ordered by counting over
// at most MSD_MAX_TREE entries, and each node builds its ancestor mask by
// walking up its parent chain in LDS.
constexpr int FIN_THREADS = 1024;  // >= the pool capacity (a power of two)

__global__ __launch_bounds__(FIN_THREADS) void k_dyn_finalize(DynPool pool, msd_tree* trees,
                                                              const int* seq_ids,
                                                              const int* d_root, int n_pool,
                                                              int N) {
  __shared__ float ks[FIN_THREADS];
  __shared__ int ki[FIN_THREADS];
  __shared__ int node_of[FIN_THREADS];
  __shared__ int kept[MSD_MAX_TREE], kdep[MSD_MAX_TREE];
  __shared__ int keep[MSD_MAX_TREE];
  __shared__ int par[MSD_MAX_TREE];
  const int sidx = blockIdx.x;
  const size_t base = (size_t)sidx * pool.cap;
  const int i = threadIdx.x;
  // past the pool: -inf keys with indices after every candidate
  ks[i] = i < n_pool ? pool.score[base + i] : -INFINITY;
  ki[i] = i;
  node_of[i] = 0;
  __syncthreads();
  // best first: "less" is better_score
  for (int k = 2; k <= FIN_THREADS; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int l = i ^ j;
      if (l > i) {
        const float si = ks[i], sl = ks[l];
        const int ii = ki[i], il = ki[l];
        const bool up = (i & k) == 0;
        if (up ? better_score(sl, il, si, ii) : better_score(si, ii, sl, il)) {
          ks[i] = sl;
          ks[l] = si;
          ki[i] = il;
          ki[l] = ii;
        }
      }
      __syncthreads();
    }
  }
  if (i < N) {
    kept[i] = ki[i];
    kdep[i] = pool.depth[base + ki[i]];
  }
  __syncthreads();
  // canonical position of kept candidate i among the N kept
  if (i < N) {
    const int c = kept[i], dc = kdep[i];
    int pos = 0;
    for (int q = 0; q < N; ++q)
      pos += (int)(kdep[q] < dc) | ((int)(kdep[q] == dc) & (int)(kept[q] < c));
    keep[pos] = c;
  }
  __syncthreads();
  if (i < N) node_of[keep[i]] = 2 + i;
  __syncthreads();
  msd_tree* t = trees + sidx;
  if (i < MSD_MAX_TREE) {
    int tok = 0, pn = -1, d = 0;
    float s = 0.f;
    if (i == 0) {
      tok = d_root[seq_ids[sidx]];
    } else if (i <= N) {
      const int c = keep[i - 1];
      const int p = pool.parent[base + c];
      // a kept node's parent is always kept (scores never increase along a
      // path) and comes earlier; the guard only keeps a malformed pool
      // inside the tree arrays
      pn = (p < 0 || p >= n_pool || node_of[p] < 2) ? 0 : node_of[p] - 1;
      tok = pool.tok[base + c];
      d = pool.depth[base + c];
      s = pool.score[base + c];
    }
    par[i] = pn;
    t->token[i] = tok;
    t->parent[i] = pn;
    t->depth[i] = d;
    t->score[i] = s;
  }
  if (i == 0) t->n_nodes = N + 1;
  __syncthreads();
  if (i < MSD_MAX_TREE) {
    uint64_t m = 0ull;
    if (i <= N) {
      int u = i;
      for (int step = 0; step < MSD_MAX_TREE && u >= 0; ++step) {
        m |= 1ull << u;
        u = (u == 0 || par[u] >= u) ? -1 : par[u];
      }
    }
    t->anc[i] = m;
  }
}

// Verify-row descriptors of one sequence's tree (one 64-thread block per
// sequence), and the tree check: tree_err[sidx] = 1 unless the tree has T
// nodes, ids in [0, vocab), a root (parent -1, depth 0, anc = bit 0) and, for
// every other node, a parent that precedes it, depth = parent's depth + 1,
// anc = parent's anc | own bit, and a token that no earlier sibling carries.
// The acceptance kernels take no decision on a call with a flagged tree.
__global__ __launch_bounds__(MSD_MAX_TREE) void k_verify_rows(
    const msd_tree* trees, const int* seq_ids, const int* d_len, int T, int vocab, Rows r,
    int* prefix, int* tree_err) {
  __shared__ int sp[MSD_MAX_TREE], sd[MSD_MAX_TREE], stk[MSD_MAX_TREE];
  __shared__ uint64_t sa[MSD_MAX_TREE];
  __shared__ int bad;
  const int sidx = blockIdx.x;
  const int i = threadIdx.x;
  const int b = seq_ids[sidx];
  const int L = d_len[b];
  const msd_tree* t = trees + sidx;
  if (i == 0) {
    prefix[sidx] = L;
    bad = t->n_nodes != T;
  }
  if (i < T) {
    sp[i] = t->parent[i];
    sd[i] = t->depth[i];
    stk[i] = t->token[i];
    sa[i] = t->anc[i];
  }
  __syncthreads();
  if (i < T) {
    bool e = stk[i] < 0 || stk[i] >= vocab;
    const int p = sp[i];
    if (i == 0) {
      e |= p != -1 || sd[0] != 0 || sa[0] != 1ull;
    } else if (p < 0 || p >= i) {
      e = true;
    } else {
      e |= sd[i] != sd[p] + 1 || sa[i] != (sa[p] | (1ull << i));
      for (int j = 1; j < i; ++j) e |= sp[j] == p && stk[j] == stk[i];
    }
    if (e) atomicOr(&bad, 1);
  }
  __syncthreads();
  if (i == 0) tree_err[sidx] = bad;
  if (i >= T) return;
  const int row = sidx * T + i;
  // caller-supplied trees: keep ids and positions inside their tables
  r.tok[row] = min(max(t->token[i], 0), vocab - 1);
  r.vis[row] = -1;
  r.pos[row] = L + min(max(t->depth[i], 0), T - 1);
  r.slot[row] = L + i;
  r.seq[row] = b;
  r.mask[row] = t->anc[i];
}



// Greedy acceptance: node j is accepted iff its parent is and its token is
// the parent's argmax; the deepest accepted node ends the path (unique since
// siblings carry distinct tokens).  One wave per sequence: the tree and the
// argmax row are staged in LDS by one lane per node, lane 0 takes the
// decisions in node order, and the lanes write the outputs.
// A call whose verify flagged any tree (tree_err) accepts nothing: every
// sequence gets an empty path, so compaction and commit leave it unchanged.
__global__ __launch_bounds__(MSD_MAX_TREE) void k_accept(const msd_tree* trees,
                                                         const int* seq_ids, int T,
                                                         const int* amax, int* path,
                                                         int* n_path, int* emitted,
                                                         int* slot_map, const int* d_len,
                                                         const int* tree_err, int n_seq) {
  __shared__ int par[MSD_MAX_TREE], tok[MSD_MAX_TREE], dep[MSD_MAX_TREE], am[MSD_MAX_TREE];
  __shared__ int pth[MSD_MAX_TREE];
  __shared__ int n_sh;
  const int sidx = blockIdx.x;
  const int j = threadIdx.x;
  const msd_tree* t = trees + sidx;
  if (any_tree_err(tree_err, n_seq)) {
    path[sidx * MSD_MAX_TREE + j] = -1;
    slot_map[sidx * MSD_MAX_TREE + j] = -1;
    emitted[sidx * MSD_MAX_TREE + j] = -1;
    if (j == 0) n_path[sidx] = 0;
    return;
  }
  if (j < T) {
    par[j] = t->parent[j];
    tok[j] = t->token[j];
    dep[j] = t->depth[j];
    am[j] = amax[(size_t)sidx * T + j];
  }
  __syncthreads();
  if (j == 0) {
    uint64_t ok = 1ull;
    int best = 0;
    for (int u = 1; u < T; ++u) {
      const int p = par[u];
      if (p < 0 || p >= u) continue;  // malformed: parents must precede children
      if (((ok >> p) & 1ull) && tok[u] == am[p]) {
        ok |= 1ull << u;
        if (dep[u] > dep[best]) best = u;
      }
    }
    // the path root .. best: its length first, then written from the end
    int n = 0;
    for (int u = best; u >= 0 && n < MSD_MAX_TREE; u = (par[u] < u) ? par[u] : -1) ++n;
    int u = best;
    for (int q = n - 1; q >= 0; --q) {
      pth[q] = u;
      u = (par[u] < u) ? par[u] : -1;
    }
    n_sh = n;
  }
  __syncthreads();
  const int n = n_sh;
  const int L = d_len[seq_ids[sidx]];
  const int u = (j < n) ? pth[j] : -1;
  path[sidx * MSD_MAX_TREE + j] = u;
  slot_map[sidx * MSD_MAX_TREE + j] = (j < n) ? L + u : -1;
  emitted[sidx * MSD_MAX_TREE + j] = (j + 1 < n) ? tok[pth[j + 1]] : ((j + 1 == n) ? am[pth[n - 1]] : -1);
  if (j == 0) n_path[sidx] = n;
}

// In place: K rows L + path[j] -> L + j and the matching V^T columns, for
// one (layer, sequence, kv head) per block; every read lands in LDS before
// the first write.
__global__ __launch_bounds__(256) void k_compact(uint16_t* kc, uint16_t* vc, int B, int KV,
                                                 int S, int hd, int n_seq, const int* seq_ids,
                                                 const int* path, const int* n_path,
                                                 const int* d_len) {
  __shared__ uint16_t ks[MSD_MAX_TREE * 128];
  __shared__ uint16_t vs[MSD_MAX_TREE * 128];
  int t = blockIdx.x;
  const int g = t % KV; t /= KV;
  const int sidx = t % n_seq;
  const int layer = t / n_seq;
  const int b = seq_ids[sidx];
  const int n = n_path[sidx];
  const int L = d_len[b];
  const int* pth = path + sidx * MSD_MAX_TREE;
  uint16_t* kb = kc + ((size_t)(layer * B + b) * KV + g) * S * hd;
  uint16_t* vb = vc + ((size_t)(layer * B + b) * KV + g) * hd * S;
  for (int idx = threadIdx.x; idx < n * hd; idx += 256) {
    const int j = idx / hd, e = idx - j * hd;
    const int src = L + pth[j];
    ks[idx] = kb[(size_t)src * hd + e];
    vs[idx] = vb[(size_t)e * S + src];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < n * hd; idx += 256) {
    const int j = idx / hd, e = idx - j * hd;
    if (pth[j] == j) continue;
    kb[(size_t)(L + j) * hd + e] = ks[idx];
    vb[(size_t)e * S + L + j] = vs[idx];
  }
}

// Accepted nodes become the next pending draft rows; the committed length
// grows by the path length and the bonus token becomes the next root.
__global__ void k_commit(const int* seq_ids, const int* path, const int* n_path,
                         const int* emitted, const uint16_t* h_tree, int T, int d,
                         uint16_t* pend_h, int* pend_next, int* pend_n, int pend_stride,
                         int* d_len, int* d_root) {
  const int sidx = blockIdx.x;
  const int j = blockIdx.y;
  const int b = seq_ids[sidx];
  const int n = n_path[sidx];
  if (j >= n) return;
  const int u = path[sidx * MSD_MAX_TREE + j];
  const uint4* src = reinterpret_cast<const uint4*>(h_tree + (size_t)(sidx * T + u) * 2 * d);
  uint4* dst = reinterpret_cast<uint4*>(pend_h + (size_t)(b * pend_stride + j) * 2 * d);
  // the split row (2d bf16, d <= 8192) in 16-byte units, every load issued
  // before the first store
  uint4 v[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int q = threadIdx.x + 256 * k;
    v[k] = 8 * q < 2 * d ? src[q] : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int q = threadIdx.x + 256 * k;
    if (8 * q < 2 * d) dst[q] = v[k];
  }
  if (threadIdx.x == 0) {
    pend_next[b * pend_stride + j] = emitted[sidx * MSD_MAX_TREE + j];
    if (j == 0) {
      pend_n[b] = n;
      d_len[b] += n;
      d_root[b] = emitted[sidx * MSD_MAX_TREE + n - 1];
    }
  }
}

__global__ void k_import_row(const uint16_t* src, int n, uint16_t* dst) {
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n; e += gridDim.x * blockDim.x) {
    dst[e] = src[e];
    dst[n + e] = 0;
  }
}

__global__ void k_set_int(int* p, int idx, const int* src, int src_idx) {
  p[idx] = src[src_idx];
}

}  // namespace

void launch_tree_init_static(void* trees, int n_seq, const int* seq_ids, const int* d_root,
                             StaticSpec sp, int T, hipStream_t st) {
  hipLaunchKernelGGL(k_tree_init_static, dim3(n_seq), dim3(64), 0, st, (msd_tree*)trees,
                     seq_ids, d_root, sp, T);
}


void launch_static_assign(void* trees, int n_seq, StaticSpec sp, int T, int parent_depth,
                          const int* topk_idx, int k, int n_round, hipStream_t st) {
  hipLaunchKernelGGL(k_static_assign, dim3(n_seq), dim3(64), 0, st, (msd_tree*)trees, sp, T,
                     parent_depth, topk_idx, k, n_round);
}

void launch_static_next(void* trees, int n_seq, const int* seq_ids, const int* d_len,
                        StaticSpec sp, int T, int depth, const int* topk_idx, int k, int n_prev,
                        int round_off, int n_round, int feat_stride, Rows r, int* prefix,
                        const float* feat, const uint16_t* E, int d, uint16_t* out,
                        hipStream_t st) {
  if (n_seq * n_round <= 0) return;
  hipLaunchKernelGGL(k_static_next, dim3(n_seq * n_round, (d + 255) / 256), dim3(256), 0, st,
                     (msd_tree*)trees, seq_ids, d_len, sp, T, depth, topk_idx, k, n_prev,
                     round_off, n_round, feat_stride, r, prefix, feat, E, d, out);
}

void launch_catchup_next(int n_seq, const int* seq_ids, const int* d_len, const int* pend_n,
                         const int* pend_next, int r_max, int pend_stride, int feat_stride,
                         Rows r, int* prefix, const uint16_t* pend_h, const uint16_t* E, int d,
                         uint16_t* out, hipStream_t st) {
  if (n_seq * r_max <= 0) return;
  hipLaunchKernelGGL(k_catchup_next, dim3(n_seq * r_max, (d + 255) / 256), dim3(256), 0, st,
                     seq_ids, d_len, pend_n, pend_next, r_max, pend_stride, feat_stride, r,
                     prefix, pend_h, E, d, out);
}

void launch_dyn_root(DynPool pool, int n_seq, const int* topk_idx, const float* topk_val,
                     const float* lse, int K, hipStream_t st) {
  hipLaunchKernelGGL(k_dyn_root, dim3(n_seq), dim3(64), 0, st, pool, topk_idx, topk_val, lse, K);
}

void launch_dyn_rows(DynPool pool, int n_seq, const int* seq_ids, const int* d_len, int K,
                     int depth, int feat_stride, Rows r, int* prefix, hipStream_t st) {
  hipLaunchKernelGGL(k_dyn_rows, dim3(n_seq), dim3(64), 0, st, pool, seq_ids, d_len, K, depth,
                     feat_stride, r, prefix);
}

void launch_dyn_expand(DynPool pool, int n_seq, const int* topk_idx, const float* topk_val,
                       const float* lse, int K, int n_pool, int exp_base, hipStream_t st) {
  hipLaunchKernelGGL(k_dyn_expand, dim3(n_seq), dim3(256), 0, st, pool, topk_idx, topk_val, lse,
                     K, n_pool, exp_base);
}

void launch_dyn_finalize(DynPool pool, void* trees, int n_seq, const int* seq_ids,
                         const int* d_root, int n_pool, int N, hipStream_t st) {
  hipLaunchKernelGGL(k_dyn_finalize, dim3(n_seq), dim3(FIN_THREADS), 0, st, pool,
                     (msd_tree*)trees, seq_ids, d_root, n_pool, N);
}

void launch_verify_rows(const void* trees, int n_seq, const int* seq_ids, const int* d_len,
                        int T, int vocab, Rows r, int* prefix, int* tree_err, hipStream_t st) {
  hipLaunchKernelGGL(k_verify_rows, dim3(n_seq), dim3(MSD_MAX_TREE), 0, st,
                     (const msd_tree*)trees, seq_ids, d_len, T, vocab, r, prefix, tree_err);
}



void launch_accept(const void* trees, int n_seq, const int* seq_ids, int T, const int* amax,
                   int* path, int* n_path, int* emitted, int* slot_map, const int* d_len,
                   const int* tree_err, hipStream_t st) {
  hipLaunchKernelGGL(k_accept, dim3(n_seq), dim3(MSD_MAX_TREE), 0, st, (const msd_tree*)trees,
                     seq_ids, T, amax, path, n_path, emitted, slot_map, d_len, tree_err, n_seq);
}

void launch_compact(uint16_t* kc, uint16_t* vc, int n_layers, int B, int KV, int S, int hd,
                    int n_seq, const int* seq_ids, const int* path, const int* n_path,
                    const int* d_len, hipStream_t st) {
  hipLaunchKernelGGL(k_compact, dim3(n_layers * n_seq * KV), dim3(256), 0, st, kc, vc, B, KV, S,
                     hd, n_seq, seq_ids, path, n_path, d_len);
}

void launch_commit(int n_seq, const int* seq_ids, const int* path, const int* n_path,
                   const int* emitted, const uint16_t* h_tree, int T, int d, uint16_t* pend_h,
                   int* pend_next, int* pend_n, int pend_stride, int* d_len, int* d_root,
                   hipStream_t st) {
  hipLaunchKernelGGL(k_commit, dim3(n_seq, MSD_MAX_TREE), dim3(256), 0, st, seq_ids, path,
                     n_path, emitted, h_tree, T, d, pend_h, pend_next, pend_n, pend_stride,
                     d_len, d_root);
}

void launch_import_row(const uint16_t* src, int n, uint16_t* dst, hipStream_t st) {
  if (n <= 0) return;
  hipLaunchKernelGGL(k_import_row, dim3((n + 255) / 256), dim3(256), 0, st, src, n, dst);
}

void launch_set_int(int* p, int idx, const int* src, int src_idx, hipStream_t st) {
  hipLaunchKernelGGL(k_set_int, dim3(1), dim3(1), 0, st, p, idx, src, src_idx);
}

}  // namespace msd
