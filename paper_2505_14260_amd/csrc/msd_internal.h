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

namespace msd {

// ---------------------------------------------------------------- GEMM ----
// Y = X W^T for a thin X (M rows) against a weight streamed from HBM.
enum Epilogue { EPI_F32 = 0, EPI_BF16 = 1, EPI_RESID = 2, EPI_SILU = 3 };

struct GemmArgs {
  const uint16_t* X;        // [M][ldx] bf16
  int ldx, M;
  const uint16_t* Wseg[3];  // [N][K] bf16 given as up to three row segments
  int seg_end[3];           // cumulative segment heights (multiples of 16)
  const uint16_t* W2;       // second weight (EPI_SILU: up projection), [N][K]
  int N, K;
  float* out_f32;           // EPI_F32 / EPI_RESID
  uint16_t* out_bf16;       // EPI_BF16 / EPI_SILU
  int ldo;
};

struct GemmScratch {
  int target_wgs;  // workgroups that keep every CU busy (tile-width choice)
};

void launch_gemm(int epi, const uint16_t* X, int ldx, int M, const uint16_t* W,
                 const uint16_t* W2, int N, int K, float* out_f32, uint16_t* out_bf16,
                 int ldo, const GemmScratch& s, hipStream_t st);
// Segmented form: the weight is the row concatenation of n_seg (<= 3)
// matrices Wseg[q] of seg_rows[q] rows each (multiples of 16).
void launch_gemm(int epi, const uint16_t* X, int ldx, int M, const uint16_t* const* Wseg,
                 const int* seg_rows, int n_seg, const uint16_t* W2, int K, float* out_f32,
                 uint16_t* out_bf16, int ldo, const GemmScratch& s, hipStream_t st);

// ----------------------------------------------------------- attention ----
struct AttnArgs {
  const uint16_t* q;      // [n_seq*nq][H*hd] bf16, rotated
  const uint16_t* kc;     // layer K cache  [B][KV][S][hd]
  const uint16_t* vc;     // layer V cache  [B][KV][hd][S]
  const int* seq_ids;     // [n_seq] absolute sequence index into the caches
  const int* prefix;      // [n_seq] fully visible prefix length
  const uint64_t* mask;   // [n_seq*nq] region masks (tree mode)
  int S, H, KV, hd, nq, n_seq, R;
  int n_chunks, chunk_keys, qtiles;
  float* part_o;          // [items][64*hd/2*...] partial outputs (tree mode)
  float* part_ml;         // [items][32][2]
  uint16_t* out;          // [n_seq*nq][H*hd] bf16
  float scale;
};

void launch_tree_attention(AttnArgs a, hipStream_t st);
void launch_causal_attention(AttnArgs a, hipStream_t st);
size_t attn_partial_floats(int n_seq, int KV, int qtiles, int n_chunks, int hd);

// ------------------------------------------------------------ row ops ----
void launch_embed(const uint16_t* E, const int* tokens, const int* vis_idx,
                  const uint16_t* visual, int rows, int d, float* x, hipStream_t st);
void launch_rmsnorm(const float* x, const uint16_t* g, int rows, int d, float eps,
                    uint16_t* y, hipStream_t st);
void launch_to_bf16(const float* x, int n, uint16_t* y, hipStream_t st);
void launch_rope_kv(const float* qkv, int rows, int H, int KV, int hd, const int* pos,
                    const int* row_seq, const int* row_slot, const float2* rope_tab,
                    uint16_t* q, uint16_t* kc, uint16_t* vc, int S, hipStream_t st);
void launch_rope_table(float2* tab, int max_pos, int hd, double theta, hipStream_t st);
void launch_fc_input(const uint16_t* h, const float* hf, const int* h_row,
                     const uint16_t* E, const int* next_tok, const uint16_t* visual,
                     int rows, int d, uint16_t* out, hipStream_t st);
void launch_visual_rows(const uint16_t* visual, const int* vis_idx, int rows, int d,
                        float* x, hipStream_t st);

// -------------------------------------------------------- selection ----
// scratch: topk_scratch_floats(rows, V) floats (8-byte aligned)
size_t topk_scratch_floats(int rows, int V);
void launch_topk(const float* logits, int rows, int V, int k, int* idx, float* val,
                 float* lse, float* scratch, hipStream_t st);

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
void launch_static_rows(const void* trees, int n_seq, const int* seq_ids, const int* d_len,
                        StaticSpec sp, int round_off, int n_round, int depth, int feat_stride,
                        Rows r, int* prefix, hipStream_t st);
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
void launch_verify_rows(const void* trees, int n_seq, const int* seq_ids, const int* d_len,
                        int T, int vocab, Rows r, int* prefix, hipStream_t st);
void launch_catchup_rows(int n_seq, const int* seq_ids, const int* d_len, const int* pend_n,
                         const int* pend_next, int r_max, int pend_stride, int feat_stride,
                         Rows r, int* prefix, hipStream_t st);
void launch_store_feat(const float* x, int rows, const int* dst, int d, float* feat,
                       hipStream_t st);
void launch_accept(const void* trees, int n_seq, const int* seq_ids, int T, const int* amax,
                   int* path, int* n_path, int* emitted, int* slot_map, const int* d_len,
                   hipStream_t st);
void launch_compact(uint16_t* kc, uint16_t* vc, int n_layers, int B, int KV, int S, int hd,
                    int n_seq, const int* seq_ids, const int* path, const int* n_path,
                    const int* d_len, hipStream_t st);
void launch_commit(int n_seq, const int* seq_ids, const int* path, const int* n_path,
                   const int* emitted, const uint16_t* h_tree, int T, int d, uint16_t* pend_h,
                   int* pend_next, int* pend_n, int pend_stride, int* d_len, int* d_root,
                   hipStream_t st);
void launch_set_int(int* p, int idx, const int* src, int src_idx, hipStream_t st);

}  // namespace msd
