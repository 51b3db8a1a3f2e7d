// Internal declarations of the gfx950 MSD library: device helpers, kernel
// argument blocks and the launchers the host orchestration calls.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

#define MSD_DEV __device__ __forceinline__

MSD_DEV float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bfloat16, round to nearest even (NaN kept quiet).
MSD_DEV uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

MSD_DEV bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Split activation rows.  A row of K values that feeds an MFMA product is
// stored as K bfloat16 "hi" values followed by K bfloat16 "lo" values with
// hi = bf16(x) and lo = bf16(x - hi): hi + lo keeps about 16 significant bits
// of x in the bytes of one float32, and W x = W hi + W lo runs on bf16 MFMA.
MSD_DEV void put_split(uint16_t* row, int K, int k, float v) {
  const uint16_t h = f2bf(v);
  row[k] = h;
  row[K + k] = f2bf(v - bf2f(h));
}
MSD_DEV float get_split(const uint16_t* row, int K, int k) {
  return bf2f(row[k]) + bf2f(row[K + k]);
}

// Workgroup barrier that orders LDS accesses only: global loads issued
// before it stay in flight.
MSD_DEV void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// True when the verify of this call flagged any of its n_seq trees.
MSD_DEV bool any_tree_err(const int* tree_err, int n_seq) {
  int e = 0;
  for (int i = 0; i < n_seq; ++i) e |= tree_err[i];
  return e != 0;
}

namespace msd {

// ---------------------------------------------------------------- GEMM ----
// Partial products of a thin X (M split rows) against a packed bf16 weight
// streamed from HBM: part[s][m][n] = sum over K-chunk s of X[m][k] * W[n][k]
// (float32).  With a second weight W2 (the SwiGLU pair) its products go to
// columns [off2, off2 + N).  The consumer sums the S chunks in order.
struct GemmArgs {
  const uint16_t* X;        // [M][ldx] split rows: hi at [k], lo at [K + k]
  int ldx, M, K;
  const uint16_t* W;        // packed (packed_elems(N, K) elements)
  const uint16_t* W2;       // second packed weight or null
  int n_tiles, nkt;         // 64-row tiles, 128-column blocks
  int S, G;                 // K chunks, workgroups per chunk
  float* part;              // partials of row 0 of this launch
  size_t part_split;        // floats between consecutive chunks (M * ldp)
  int ldp, off2;            // floats between rows; column offset of W2's products
  float* sink;              // 1 KB written by padded rows
};

struct GemmPlan {
  int MT, nkb, S, G, nw, n_tiles, nkt, ldp, off2;
  int pair;  // 2, 3 or 4: K chunks per workgroup (S counts their groups); 0: one
  int fk;    // > 0: all of K per workgroup for fk tiles (S = 1)
  int per;   // tiles per workgroup
  int ms;    // 33-64 rows as two 32-row halves (MT, S and G of one half)
};

struct GemmScratch {
  int target_wgs;                // workgroups per launch
  hipEvent_t ev_start, ev_stop;  // when set: recorded around the kernel itself
};

// Elements of a packed [N][K] weight (64-row tiles x 128-column blocks).
size_t packed_elems(int N, int K);
// Packs the row-major bf16 [N][K] src into dst (packed_elems(N, K) elements).
void launch_pack(const uint16_t* src, int N, int K, uint16_t* dst, hipStream_t st);
// Row-major bf16 [N][K] back from the packed layout (K a multiple of 8).
void launch_unpack(const uint16_t* src, int N, int K, uint16_t* dst, hipStream_t st);
GemmPlan plan_gemm(int M, int N, int K, int nw, int target_wgs);
// floats of partials for M rows (M <= 64 per launch)
size_t gemm_part_floats(int M, int N, int K, int nw, int target_wgs);
// Diagnostic: reads spans * stream_span_bytes() bytes of buf with the weight
// stream's access pattern on wgs workgroups (sink: wgs words, never written
// for zero-filled buffers).
size_t stream_span_bytes();
void launch_stream_read(const uint16_t* buf, size_t spans, int wgs, unsigned* sink,
                        hipStream_t st);
void launch_gemm(const uint16_t* X, int ldx, int M, const uint16_t* W, const uint16_t* W2, int N,
                 int K, float* part, float* sink, const GemmScratch& sc, hipStream_t st);

// Partial sums as seen by a consumer: value(m, n) = sum_s p[s*split + m*ld + n];
// the second weight's products are at column n + off2.
struct Parts {
  const float* p;
  int S;
  size_t split;
  int ld, off2;
};

// Per-row sums of squares come in blocks of SSQ_BLOCK features.
// Row width limit of the whole-row kernels (four 16-byte units per thread).
constexpr int MAX_D_MODEL = 8192;
constexpr int SSQ_BLOCK = 1024;
inline int ssq_blocks(int d) { return (d + SSQ_BLOCK - 1) / SSQ_BLOCK; }

// Per-row RMS of the un-normalised GEMM input: ssq[row][0..nblk) are sums of
// x^2 over blocks of SSQ_BLOCK features (ssq == null: no scaling).
struct RowNorm {
  const float* ssq;
  int nblk, d;
  float eps;
};

// ----------------------------------------------------------- attention ----
constexpr int ATT_MAX_SEQ = 8;
#ifndef MSD_TREE_WAVES
#define MSD_TREE_WAVES 4
#endif
constexpr int TREE_WAVES = MSD_TREE_WAVES;  // waves per tree-attention workgroup
// key chunks per (sequence, kv head, query tile): the workgroup that
// finishes an item's last chunk merges at most this many partials
constexpr int ATT_MAX_CHUNKS = 8;
// tree-attention workgroups a pass aims for (about eight waves per CU)
constexpr int ATT_TARGET_WGS = 256 * 8 / TREE_WAVES;
struct AttnArgs {
  const uint16_t* q;      // [n_seq*nq] split rows of H*hd, rotated
  const uint16_t* kc;     // layer K cache  [B][KV][S][hd]
  const uint16_t* vc;     // layer V cache  [B][KV][hd][S]
  int seq[ATT_MAX_SEQ];   // absolute sequence index into the caches, per call slot
  int prefix[ATT_MAX_SEQ];  // fully visible prefix length, per call slot
  int keys[ATT_MAX_SEQ];  // tree mode: slots [prefix, keys) are the masked region;
                          // no slot at or past keys is read
  const uint64_t* mask;   // [n_seq*nq] region masks (tree mode)
  int S, H, KV, hd, nq, n_seq;
  int n_chunks, chunk_keys, qtiles;  // chunk_keys: multiple of 128 (tree mode)
  int xrep;               // XCDs per (sequence, kv head) pair (set by the launcher)
  float* part_o;          // [items][32*hd] float16 partial outputs (tree mode, n_chunks > 1)
  float* part_ml;         // [items][32][2]
  int* att_cnt;           // [items] chunk arrivals per XCD (zero between launches)
  int* place_err;         // set to 1 when an item's chunks ran on more than one XCD
  uint16_t* out;          // [n_seq*nq] split rows of H*hd
  float scale;
};

// ev0/ev1 (optional): events recorded by the launches themselves, before
// the attention kernel and after the last kernel of the pass.
void launch_tree_attention(AttnArgs a, hipStream_t st, hipEvent_t ev0 = nullptr,
                           hipEvent_t ev1 = nullptr);
void launch_causal_attention(AttnArgs a, hipStream_t st);
size_t attn_partial_floats(int n_seq, int KV, int qtiles, int n_chunks, int hd);

// ------------------------------------------------------------ row ops ----
void launch_embed(const uint16_t* E, const int* tokens, const int* vis_idx,
                  const uint16_t* visual, int rows, int d, float* x, hipStream_t st);
// x = (mode 1) sum of parts, (mode 2) x + sum of parts, (mode 0) x; then
// xn = rmsnorm(x) * g when g, xb = x when xb (split rows of d).
enum { RN_KEEP = 0, RN_SET = 1, RN_ADD = 2 };
void launch_resid_norm(Parts pt, int col0, int rows, int d, int mode, float* x,
                       const uint16_t* g, float eps, uint16_t* xn, uint16_t* xb, hipStream_t st);
// act = silu(gate) * up (split rows of F)
void launch_silu(Parts pt, RowNorm rn, int rows, int F, uint16_t* act, hipStream_t st);
// Elementwise form: x updated as above, xg = x * g when xg, xb = x when xb
// (split rows of d), ssq[row][blk] = sum of x^2 over feature block blk
// (256 wide).
// feat: when given, row r of the new x is also copied to feat row dst[r]
// (dst[r] < 0: no copy), the draft's feature store.
void launch_resid(Parts pt, int rows, int d, int mode, float* x, const uint16_t* g, uint16_t* xg,
                  uint16_t* xb, float* ssq, hipStream_t st, const int* dst = nullptr,
                  float* feat = nullptr);
void launch_rope_kv(Parts qkv, RowNorm rn, int rows, int H, int KV, int hd, const int* pos,
                    const int* row_seq, const int* row_slot, const float2* rope_tab,
                    uint16_t* q, uint16_t* kc, uint16_t* vc, int S, hipStream_t st);
void launch_rope_table(float2* tab, int max_pos, int hd, double theta, hipStream_t st);
// out[row] = split row of [h | e] (2d values); h rows are split rows of d
// (target features) when h, else float32 rows of hf (draft features).
void launch_fc_input(const uint16_t* h, const float* hf, const int* h_row, const uint16_t* E,
                     const int* next_tok, const uint16_t* visual, int rows, int d, uint16_t* out,
                     hipStream_t st);
void launch_visual_rows(const uint16_t* visual, const int* vis_idx, int rows, int d,
                        float* x, hipStream_t st);
// x rows with vis_idx >= 0 = the split rows h (the target features).
void launch_visual_feature_rows(const uint16_t* h, const int* vis_idx, int rows, int d, float* x,
                                hipStream_t st);

// -------------------------------------------------------- selection ----
// scratch: topk_scratch_floats(rows, V) floats (8-byte aligned).  The
// logits are the summed parts; when logits_out is given they are also
// written there ([rows][V]).
size_t topk_scratch_floats(int rows, int V);
void launch_topk(Parts logits, int rows, int V, int k, int* idx, float* val, float* lse,
                 float* logits_out, float* scratch, hipStream_t st);

// ---------------------------------------------------- tree / accept ----
// Row descriptors of one forward step (device arrays, one entry per row).
struct Rows {
  int* tok;        // input token (verify) / next token for f_down (draft)
  int* vis;        // visual row index or -1
  int* pos;        // RoPE position
  int* slot;       // cache slot (-1: do not write)
  int* seq;        // absolute sequence index
  int* hrow;       // feature row for the draft input
  uint64_t* mask;  // region mask (tree attention)
  int* dst;        // destination feature slot (draft expansions)
};

// Static tree template kept on the device (node 0 = root).
struct StaticSpec {
  int* parent;      // [T]
  int* rank;        // [T]
  int* depth;       // [T]
  uint64_t* anc;    // [T]
  int* exp_idx;     // [T] expansion index or -1
  uint64_t* exp_mask;  // [T] mask over expansion indices
  int* pslot;       // [T] feature slot of the node's parent (0 = root feature)
  int* round_nodes; // [T] nodes expanded per round, concatenated by depth
  int* round_pos;   // [T] position of a node within its expansion round
};

struct DynPool {
  int* parent;     // [B][P] pool index of the parent, -1 = root
  int* tok;
  int* depth;
  float* score;
  int* exp_idx;    // expansion index, -1 if never expanded
  uint64_t* mask;  // expansion-ancestor mask
  int* frontier;   // [B][K]
  int cap;         // P
};

void launch_tree_init_static(void* trees, int n_seq, const int* seq_ids, const int* d_root,
                             StaticSpec sp, int T, hipStream_t st);
// Round `depth` of a static tree: the depth's tokens from the previous
// round's top-k, the round's row descriptors and f_down inputs.
void launch_static_next(void* trees, int n_seq, const int* seq_ids, const int* d_len,
                        StaticSpec sp, int T, int depth, const int* topk_idx, int k, int n_prev,
                        int round_off, int n_round, int feat_stride, Rows r, int* prefix,
                        const float* feat, const uint16_t* E, int d, uint16_t* out,
                        hipStream_t st);
// Catch-up rows (pending draft rows) and their f_down inputs.
void launch_catchup_next(int n_seq, const int* seq_ids, const int* d_len, const int* pend_n,
                         const int* pend_next, int r_max, int pend_stride, int feat_stride,
                         Rows r, int* prefix, const uint16_t* pend_h, const uint16_t* E, int d,
                         uint16_t* out, hipStream_t st);
// Root rows of a draft tree: x = each sequence's last feature, xb the same
// as split rows.
void launch_root_feat(int n_seq, const int* seq_ids, const float* feat, int feat_stride, int d,
                      float* x, uint16_t* xb, hipStream_t st);
void launch_static_assign(void* trees, int n_seq, StaticSpec sp, int T, int parent_depth,
                          const int* topk_idx, int k, int n_round, hipStream_t st);
void launch_dyn_root(DynPool pool, int n_seq, const int* topk_idx, const float* topk_val,
                     const float* lse, int K, hipStream_t st);
void launch_dyn_rows(DynPool pool, int n_seq, const int* seq_ids, const int* d_len, int K,
                     int depth, int feat_stride, Rows r, int* prefix, hipStream_t st);
void launch_dyn_expand(DynPool pool, int n_seq, const int* topk_idx, const float* topk_val,
                       const float* lse, int K, int n_pool, int exp_base, hipStream_t st);
void launch_dyn_finalize(DynPool pool, void* trees, int n_seq, const int* seq_ids,
                         const int* d_root, int n_pool, int N, hipStream_t st);
// Verify rows of each tree; tree_err[sidx] = 1 when the tree is malformed.
void launch_verify_rows(const void* trees, int n_seq, const int* seq_ids, const int* d_len,
                        int T, int vocab, Rows r, int* prefix, int* tree_err, hipStream_t st);
// Greedy acceptance; when any tree_err[0..n_seq) is set, every path is empty.
void launch_accept(const void* trees, int n_seq, const int* seq_ids, int T, const int* amax,
                   int* path, int* n_path, int* emitted, int* slot_map, const int* d_len,
                   const int* tree_err, hipStream_t st);
// Speculative sampling acceptance (k_sample.hip): same outputs as launch_accept.
void launch_accept_sample(const void* trees, int n_seq, const int* seq_ids, int T,
                          const float* logits, int V, float inv_t, uint64_t seed, int* path,
                          int* n_path, int* emitted, int* slot_map, const int* d_len,
                          const int* tree_err, hipStream_t st);
void launch_compact(uint16_t* kc, uint16_t* vc, int n_layers, int B, int KV, int S, int hd,
                    int n_seq, const int* seq_ids, const int* path, const int* n_path,
                    const int* d_len, hipStream_t st);
void launch_commit(int n_seq, const int* seq_ids, const int* path, const int* n_path,
                   const int* emitted, const uint16_t* h_tree, int T, int d, uint16_t* pend_h,
                   int* pend_next, int* pend_n, int pend_stride, int* d_len, int* d_root,
                   hipStream_t st);
// dst = split row of the bf16 row src[0..n) (lo = 0): an imported feature
void launch_import_row(const uint16_t* src, int n, uint16_t* dst, hipStream_t st);
void launch_set_int(int* p, int idx, const int* src, int src_idx, hipStream_t st);

// ------------------------------------------------------------ training ----
// Kernels of the draft-head training step (k_train.hip), float32, row-major,
// R = n - 1 rows.
// visual_feature: visual rows take the target feature (the Visual Feature
// variant) instead of their embedding
void tr_inputs(const uint16_t* h, const uint16_t* E, const int* tok, const int* vis_idx,
               const uint16_t* visual, int n, int d, int visual_feature, float* H, float* X0,
               float* E0, hipStream_t st);
void tr_visual_rows(float* F, const float* E0, const int* vis_idx, int R, int d, hipStream_t st);
void tr_zero_visual(float* dF, const int* vis_idx, int R, int d, hipStream_t st);
void tr_rmsnorm(const float* X, const float* g, float eps, int R, int d, float* Y, float* rstd,
                hipStream_t st);
// dX += the input gradient, dg += the gain gradient
void tr_rmsnorm_bwd(const float* X, const float* g, const float* rstd, const float* dY, int R,
                    int d, float* dX, float* dg, hipStream_t st);
void tr_rope(float* X, int R, int nh, int hd, const float2* tab, int dir, hipStream_t st);
void tr_softmax(float* S, int R, int heads, float scale, hipStream_t st);
void tr_softmax_bwd(const float* P, float* dP, int R, int heads, float scale, hipStream_t st);
void tr_silu(const float* G, const float* U, size_t n, float* Mx, hipStream_t st);
void tr_silu_bwd(const float* G, const float* U, const float* dM, size_t n, float* dG, float* dU,
                 hipStream_t st);
void tr_reg(const float* D, const float* H, int R, int d, float* dD, float* reg, hipStream_t st);
void tr_ce(float* Ld, const float* Lt, int R, int V, float w, float* ce, hipStream_t st);
void tr_adamw(float* w, const float* gsum, float* m, float* v, size_t n, float gscale, float lr,
              float c1, float c2, float b1, float b2, float eps, uint16_t* wb, hipStream_t st);
void tr_widen(const uint16_t* src, size_t n, float* dst, hipStream_t st);
void tr_fill(float* p, size_t n, float v, hipStream_t st);

}  // namespace msd
