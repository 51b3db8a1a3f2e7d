// C ABI of the MSD decode path (see include/msd.h): buffer planning, the
// per-call orchestration of the HIP kernels and the host-side sequence state.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <string>
#include <vector>

#include <rocblas/rocblas.h>

#include "../../include/msd.h"
#include "msd_internal.h"

using namespace msd;

// Scratch of msd_verify_noalloc: GEMM split-K partials, attention partials
// and top-k scratch of one verify call.  One copy per GPU, held until the
// process ends.  Host code never uses this name as an address: it takes the
// device address from hipGetSymbolAddress (noalloc_scratch below).
static __device__ __align__(256) float scratch[MSD_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES];  // device address of `scratch` per device

// The device address of this device's `scratch` (resolved once per device,
// with that device current), or an error.
hipError_t noalloc_scratch(int dev, void** out) {
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

namespace {

struct LayerW {
  const uint16_t *wq, *wk, *wv, *wo, *wg, *wu, *wd, *n1, *n2;
};

LayerW to_layer(const msd_layer_weights& l) {
  return {(const uint16_t*)l.wq, (const uint16_t*)l.wk, (const uint16_t*)l.wv,
          (const uint16_t*)l.wo, (const uint16_t*)l.w_gate, (const uint16_t*)l.w_up,
          (const uint16_t*)l.w_down, (const uint16_t*)l.attn_norm, (const uint16_t*)l.ffn_norm};
}

// A layer's GEMM weights in the packed layout (q|k|v fused).
struct PackedLayer {
  const uint16_t *qkv, *o, *g, *u, *d;
};

// Element offsets of every packed weight in the caller's weight arena:
// per target layer q|k|v, o, gate, up, down; the draft layer; f_down; LM head.
struct WeightLayout {
  std::vector<size_t> layer_off;  // n_layers + 1 (draft last), start of each layer
  size_t qkv, o, g, u, d;         // sizes of one layer's packed matrices
  size_t fc_off, lm_off, total;
};

WeightLayout weight_layout(const msd_model_desc& m) {
  WeightLayout w;
  const int d = m.d_model, hd = m.head_dim, H = m.n_heads, KV = m.n_kv_heads, F = m.ffn_dim;
  w.qkv = packed_elems(H * hd, d) + 2 * packed_elems(KV * hd, d);
  w.o = packed_elems(d, H * hd);
  w.g = w.u = packed_elems(F, d);
  w.d = packed_elems(d, F);
  const size_t per = w.qkv + w.o + w.g + w.u + w.d;
  size_t off = 0;
  for (int l = 0; l <= m.n_layers; ++l) {
    w.layer_off.push_back(off);
    off += per;
  }
  w.fc_off = off;
  off += packed_elems(d, 2 * d);
  w.lm_off = off;
  off += packed_elems(m.vocab, d);
  w.total = off;
  return w;
}

constexpr int MSD_MAX_BATCH_ARGS = ATT_MAX_SEQ;
constexpr int PEND = MSD_MAX_TREE;      // pending draft rows per sequence
constexpr int FEAT = MSD_MAX_TREE + 1;  // draft feature slots per sequence
constexpr int TOPK = 16;
constexpr int MAX_VOCAB = 262144;  // 128 top-k slices of 2048 logits
constexpr int POOL = 1024;              // dynamic-tree candidates per sequence
constexpr int STAGE_INTS = 1 << 16;
constexpr int ACC_BACK_INTS = 8 * MSD_MAX_TREE + 8 + 8 + 1;
// GEMM launch shape: about one workgroup per CU streams best (more
// concurrent weight streams per CU lower the achieved HBM bandwidth).
constexpr int GEMM_WGS = 256;
constexpr int CHUNK = 64;         // rows per weight-streaming GEMM launch
constexpr int BIG_CHUNK = 1024;   // rows per many-row (rocBLAS) GEMM launch
constexpr size_t BLAS_WS_BYTES = (size_t)32 << 20;  // rocBLAS's workspace
// rocBLAS products whose hi and lo results together take at most this many
// bytes (fewer than BIG_CHUNK rows), or BLAS_ONE_PRODUCT_FULL_BYTES (launches
// of BIG_CHUNK rows), run as one product over 2M interleaved rows (see
// blas_gemm)
constexpr size_t BLAS_ONE_PRODUCT_BYTES = (size_t)192 << 20;
constexpr size_t BLAS_ONE_PRODUCT_FULL_BYTES = (size_t)128 << 20;
// Tree passes (verify, draft) over more rows than BIG_MIN_ROWS, and causal
// passes (prompts, training sequences) over more than PROMPT_BIG_MIN_ROWS,
// run their GEMMs on rocBLAS in launches of up to BIG_CHUNK rows (bf16
// products with float32 results against row-major weights; a last launch of
// CHUNK rows or fewer takes the weight-streaming kernels).  Shorter passes
// run as weight-streaming launches of CHUNK rows.  7B-shaped prompts: 128
// rows 9.0 ms streamed against 10.0 ms on rocBLAS, 192 rows 13.5 against
// 11.1 ms, 256 rows 17.9 against 12.5 ms.  Target tree passes take the
// prompt threshold when their output, gate, up and down products can read
// the caller's row-major matrices in place (msd_use_caller_weights): the
// Qwen2.5-VL-7B-shaped batch-4 verify (244 rows), whose 64-row launches
// stream every weight four times, 17.2 -> 12.4 ms; unpacking the
// weights on every verify instead would cost more than it saves (17.9 ms).
constexpr int BIG_MIN_ROWS = 256;
constexpr int PROMPT_BIG_MIN_ROWS = 128;

// Rows per GEMM launch for a pass over `rows` rows (causal: a prompt pass;
// in_place: the target's row-major matrices are readable in place).
int row_chunk(int rows, bool causal, bool in_place) {
  return rows > (causal || in_place ? PROMPT_BIG_MIN_ROWS : BIG_MIN_ROWS) ? BIG_CHUNK : CHUNK;
}

// Bump allocator over the workspace (also used to size it).
struct Carver {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t n) {
    off = (off + 255) & ~(size_t)255;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

struct Plan {
  int rows_max, lrows, ld_qkv;
  int att_items;  // tree-attention items (sequence, kv head, query tile)
  size_t attn_floats, part_floats;
  size_t wrm_elems;  // row-major copy of the largest layer weight (0: no rocBLAS path)
};

Plan make_plan(const msd_model_desc& m, const msd_limits& lim) {
  Plan p;
  p.rows_max = std::max(lim.max_prompt, lim.max_batch * MSD_MAX_TREE);
  p.lrows = lim.max_batch * MSD_MAX_TREE;
  p.ld_qkv = (m.n_heads + 2 * m.n_kv_heads) * m.head_dim;
  const int G = m.n_heads / m.n_kv_heads;
  const int qtiles = (MSD_MAX_TREE * G + 31) / 32;
  p.att_items = lim.max_batch * m.n_kv_heads * qtiles;
  p.attn_floats =
      attn_partial_floats(lim.max_batch, m.n_kv_heads, qtiles, ATT_MAX_CHUNKS, m.head_dim);
  // GEMM partials of one launch of up to 64 rows, for the largest weight of
  // the model (the plans change at 16, 32 and 64 rows; within each class the
  // partials grow with the rows)
  const int d = m.d_model, F = m.ffn_dim, hh = m.n_heads * m.head_dim;
  p.part_floats = 0;
  for (int mm : {16, 32, 64}) {
    mm = std::min(mm, p.rows_max);
    const size_t cand[6] = {gemm_part_floats(mm, p.ld_qkv, d, 1, GEMM_WGS),
                            gemm_part_floats(mm, d, hh, 1, GEMM_WGS),
                            gemm_part_floats(mm, F, d, 2, GEMM_WGS),
                            gemm_part_floats(mm, d, F, 1, GEMM_WGS),
                            gemm_part_floats(mm, d, 2 * d, 1, GEMM_WGS),
                            gemm_part_floats(mm, m.vocab, d, 1, GEMM_WGS)};
    p.part_floats = std::max(p.part_floats, *std::max_element(cand, cand + 6));
  }
  // full products of one rocBLAS launch (every GEMM but the LM head, which
  // always runs in CHUNK-row launches), in either form of blas_gemm
  p.wrm_elems = 0;
  if (lim.max_prompt > PROMPT_BIG_MIN_ROWS || lim.max_batch * MSD_MAX_TREE > BIG_MIN_ROWS) {
    const size_t big = std::min(BIG_CHUNK, p.rows_max);
    auto ldp = [](int N, int nw) { return (size_t)(N + 63) / 64 * 64 * nw; };
    const size_t w = std::max({ldp(p.ld_qkv, 1), ldp(d, 1), ldp(F, 2)});
    p.part_floats = std::max(p.part_floats, big * w);
    p.part_floats = std::max(p.part_floats,
                             std::min(2 * big * w, BLAS_ONE_PRODUCT_BYTES / sizeof(float)));
    p.wrm_elems = std::max({(size_t)p.ld_qkv * d, (size_t)d * hh, (size_t)F * d, (size_t)d * 2 * d});
  }
  return p;
}

}  // namespace

// Draft-head training state (Sec. 4.2).  Float32 master copies of the
// draft's parameters (f_down, the layer's seven matrices, its two norm gains,
// in that order), their gradient sums and AdamW moments; float32 activations
// of one training pass of up to max_prompt - 1 rows; a float32 copy of the
// frozen LM head.  The contractions run as rocBLAS float32 GEMMs on the
// context's stream, everything else in k_train.hip.
constexpr int TRAIN_PARAMS = 10;
constexpr float TRAIN_CLS_WEIGHT = 0.1f;  // weight of the token term
constexpr float ADAM_B1 = 0.9f, ADAM_B2 = 0.999f, ADAM_EPS = 1e-8f;

struct TrainState {
  rocblas_handle blas = nullptr;
  int Rmax = 0;
  size_t off[TRAIN_PARAMS + 1] = {};  // float offsets of the parameters
  float *w = nullptr, *g = nullptr, *m = nullptr, *v = nullptr;
  uint16_t* wb = nullptr;             // bf16 copy of w (inference packing, norm gains)
  float* lm = nullptr;                // [V][d]
  float *H, *X0, *E0, *F, *A1, *r1, *Q, *K, *V, *S, *dP, *O, *X1, *A2, *r2, *G, *U, *Mx, *D;
  float *Ld, *Lt, *dD, *dMx, *dG, *dU, *dA2, *dX1, *dO, *dQ, *dK, *dV, *dA1, *dF;
  float *reg, *ce;
  std::vector<void*> allocs;
  double rows = 0;                    // rows accumulated since the last update
  int steps = 0;                      // updates applied
};

struct msd_ctx {
  msd_model_desc m;
  msd_limits lim;
  Plan plan;
  hipStream_t st;
  std::vector<LayerW> layers;
  LayerW dlayer;
  std::vector<PackedLayer> players;
  PackedLayer pdlayer;
  const uint16_t *embed, *final_norm, *lm_p, *fc_p;
  uint16_t *tk, *tv, *dk, *dv;
  // workspace
  float* x;
  // activation rows: split rows (bf16 hi + lo) for every MFMA input
  uint16_t *xn, *xb, *fcin, *q, *ao, *act, *h;
  float* part;
  float* sink;          // GEMM rows past M
  uint16_t* wrm;        // two row-major bf16 weight slots (rocBLAS prompt GEMMs)
  const uint16_t* wrm_src[2] = {nullptr, nullptr};  // packed weight each slot holds
  void* blas_ws;        // rocBLAS's workspace (BLAS_WS_BYTES)
  rocblas_handle blas = nullptr;  // prompt GEMMs, when plan.wrm_elems > 0
  // the target's prompt GEMMs read the caller's row-major matrices (layers)
  // instead of unpacking their packed copies (msd_use_caller_weights)
  bool caller_w = false;
  ~msd_ctx() {
    if (blas) (void)rocblas_destroy_handle(blas);
  }
  float* ssq;
  Rows rows;
  int *nxt, *prefix, *seq_ids;
  int *d_len, *d_root, *pend_n, *pend_next;
  uint16_t* pend_h;
  float* dfeat;
  int *acc_path, *acc_n, *acc_emit, *acc_slot, *feat_idx;
  int* tree_err;  // per call slot: the last verify found the tree malformed
  int* tk_idx;
  float *tk_val, *tk_lse;
  StaticSpec sp;
  DynPool pool;
  GemmScratch gs;
  float *att_po, *att_ml, *tk_scratch;
  int* att_cnt;
  int* att_place;  // tree attention merged chunks that ran on different XCDs
  float2* rope;
  int visual_input = MSD_DRAFT_VISUAL_EMBEDDING;  // draft input of visual prompt rows
  TrainState* tr = nullptr;  // draft-head training state (from the first training call)
  int device;            // the GPU current at msd_create
  float* noalloc_base;   // that GPU's copy of `scratch`
  // host
  int* stage;  // pinned staging
  std::vector<int> L, pend, ready;
  std::vector<int> seq_ids_h;  // what c->seq_ids holds (empty: unknown)
  // attention bounds of the next passes per call slot: slots below att_pre
  // are visible to every row, [att_pre, att_keys) through the row masks
  int att_pre[MSD_MAX_BATCH_ARGS];
  int att_keys[MSD_MAX_BATCH_ARGS];
  std::string err;
  // static spec cache
  std::vector<int> sp_parent, sp_rank;
  std::vector<int> round_off, round_n, round_k, round_exp_end;
  int sp_T = 0, sp_D = 0;
  // the last msd_verify not yet followed by an acceptance (verified_T == 0: none)
  int verified_T = 0;
  std::vector<int> verified_seqs;
  // optional per-GEMM event trace (msd_trace_enable)
  struct TraceRec {
    int epi, M, N, K;
    hipEvent_t a, b;
  };
  std::vector<TraceRec> trace;
  std::vector<hipEvent_t> ev_pool;
  size_t trace_cap = 0;
  bool tracing = false;
  int trace_kinds = 0;  // bit per epilogue kind
};

namespace {

std::string g_err;

int fail(msd_ctx* c, int code, const std::string& msg) {
  if (c)
    c->err = msg;
  else
    g_err = msg;
  return code;
}

#define HIPC(c, expr)                                                              \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess)                                                          \
      return fail(c, MSD_ERR_HIP, std::string(#expr ": ") + hipGetErrorString(e_)); \
  } while (0)

#define LAUNCHED(c)                                                                   \
  do {                                                                                \
    hipError_t e_ = hipGetLastError();                                                \
    if (e_ != hipSuccess)                                                             \
      return fail(c, MSD_ERR_HIP, std::string("kernel launch: ") + hipGetErrorString(e_)); \
  } while (0)

#define TRY(x)              \
  do {                      \
    int r_ = (x);           \
    if (r_ != MSD_OK) return r_; \
  } while (0)

size_t kv_bytes(const msd_model_desc& m, const msd_limits& lim, int layers) {
  return (size_t)layers * lim.max_batch * m.n_kv_heads * (size_t)lim.max_seq * m.head_dim * 2;
}

// Lays out the workspace (base == nullptr: only measures it).
size_t carve(msd_ctx* c, const msd_model_desc& m, const msd_limits& lim, char* base) {
  const Plan p = make_plan(m, lim);
  Carver cv{base};
  const int d = m.d_model, R = p.rows_max, B = lim.max_batch;
  msd_ctx tmp;
  msd_ctx* t = c ? c : &tmp;
  t->x = cv.take<float>((size_t)R * d);
  t->xn = cv.take<uint16_t>((size_t)R * 2 * d);
  t->xb = cv.take<uint16_t>((size_t)R * 2 * d);
  t->fcin = cv.take<uint16_t>((size_t)R * 4 * d);
  t->part = cv.take<float>(p.part_floats);
  t->sink = cv.take<float>(256);
  t->wrm = p.wrm_elems ? cv.take<uint16_t>(2 * p.wrm_elems) : nullptr;
  t->blas_ws = p.wrm_elems ? (void*)cv.take<char>(BLAS_WS_BYTES) : nullptr;
  t->ssq = cv.take<float>((size_t)R * ssq_blocks(d));
  t->q = cv.take<uint16_t>((size_t)R * 2 * m.n_heads * m.head_dim);
  t->ao = cv.take<uint16_t>((size_t)R * 2 * m.n_heads * m.head_dim);
  t->act = cv.take<uint16_t>((size_t)R * 2 * m.ffn_dim);
  t->h = cv.take<uint16_t>((size_t)R * 2 * d);
  t->rows.tok = cv.take<int>(R);
  t->rows.vis = cv.take<int>(R);
  t->rows.pos = cv.take<int>(R);
  t->rows.slot = cv.take<int>(R);
  t->rows.seq = cv.take<int>(R);
  t->rows.hrow = cv.take<int>(R);
  t->rows.dst = cv.take<int>(R);
  t->rows.mask = cv.take<uint64_t>(R);
  t->nxt = cv.take<int>(R);
  t->prefix = cv.take<int>(B);
  t->seq_ids = cv.take<int>(B);
  t->d_len = cv.take<int>(B);
  t->d_root = cv.take<int>(B);
  t->pend_n = cv.take<int>(B);
  t->pend_next = cv.take<int>((size_t)B * PEND);
  t->pend_h = cv.take<uint16_t>((size_t)B * PEND * 2 * d);
  t->dfeat = cv.take<float>((size_t)B * FEAT * d);
  t->acc_path = cv.take<int>((size_t)B * MSD_MAX_TREE);
  // what the host reads after an acceptance, back to back so that one copy
  // brings it: acc_emit [8][MSD_MAX_TREE], acc_n [8], tree_err [8],
  // att_place [1] (at most eight sequences per context)
  int* const accb = cv.take<int>(ACC_BACK_INTS);
  t->acc_emit = accb;
  t->acc_n = accb + 8 * MSD_MAX_TREE;
  t->tree_err = t->acc_n + 8;
  t->att_place = t->tree_err + 8;
  t->acc_slot = cv.take<int>((size_t)B * MSD_MAX_TREE);
  t->feat_idx = cv.take<int>(B);
  t->tk_idx = cv.take<int>((size_t)p.lrows * TOPK);
  t->tk_val = cv.take<float>((size_t)p.lrows * TOPK);
  t->tk_lse = cv.take<float>(p.lrows);
  t->sp.parent = cv.take<int>(MSD_MAX_TREE);
  t->sp.rank = cv.take<int>(MSD_MAX_TREE);
  t->sp.depth = cv.take<int>(MSD_MAX_TREE);
  t->sp.anc = cv.take<uint64_t>(MSD_MAX_TREE);
  t->sp.exp_idx = cv.take<int>(MSD_MAX_TREE);
  t->sp.exp_mask = cv.take<uint64_t>(MSD_MAX_TREE);
  t->sp.pslot = cv.take<int>(MSD_MAX_TREE);
  t->sp.round_nodes = cv.take<int>(MSD_MAX_TREE);
  t->sp.round_pos = cv.take<int>(MSD_MAX_TREE);
  t->pool.cap = POOL;
  t->pool.parent = cv.take<int>((size_t)B * POOL);
  t->pool.tok = cv.take<int>((size_t)B * POOL);
  t->pool.depth = cv.take<int>((size_t)B * POOL);
  t->pool.score = cv.take<float>((size_t)B * POOL);
  t->pool.exp_idx = cv.take<int>((size_t)B * POOL);
  t->pool.mask = cv.take<uint64_t>((size_t)B * POOL);
  t->pool.frontier = cv.take<int>((size_t)B * TOPK);
  t->att_po = cv.take<float>(p.attn_floats);
  t->att_ml = cv.take<float>(p.attn_floats / m.head_dim * 2 + 64);
  t->att_cnt = cv.take<int>(p.att_items);
  t->rope = cv.take<float2>((size_t)lim.max_seq * (m.head_dim / 2));
  t->tk_scratch = cv.take<float>(topk_scratch_floats(p.lrows, m.vocab));
  return cv.off + 256;
}

int check_desc(const msd_model_desc* m, const msd_limits* lim, msd_ctx* c) {
  if (!m || !lim) return fail(c, MSD_ERR_INVALID_ARG, "null model or limits");
  if (m->n_layers <= 0 || m->d_model <= 0 || m->n_heads <= 0 || m->n_kv_heads <= 0 ||
      m->n_heads % m->n_kv_heads || m->ffn_dim <= 0 || m->vocab < TOPK)
    return fail(c, MSD_ERR_INVALID_ARG, "bad model shape");
  if (m->vocab > MAX_VOCAB) return fail(c, MSD_ERR_INVALID_ARG, "vocabulary larger than 262144");
  if (m->head_dim != 128 && m->head_dim != 64)
    return fail(c, MSD_ERR_INVALID_ARG, "head_dim must be 64 or 128");
  if (m->d_model % 8 || m->ffn_dim % 8)
    return fail(c, MSD_ERR_INVALID_ARG, "d_model and ffn_dim must be multiples of 8");
  if (m->d_model > MAX_D_MODEL) return fail(c, MSD_ERR_INVALID_ARG, "d_model larger than 8192");
  if (m->n_heads / m->n_kv_heads > 16)
    return fail(c, MSD_ERR_INVALID_ARG, "query group larger than 16");
  {
    // the weight-streaming GEMMs address a packed matrix with 32-bit byte
    // offsets
    const int d = m->d_model, hd = m->head_dim, F = m->ffn_dim;
    const int qkv = (m->n_heads + 2 * m->n_kv_heads) * hd, hh = m->n_heads * hd;
    const int shapes[6][2] = {{qkv, d}, {d, hh}, {F, d}, {d, F}, {d, 2 * d}, {m->vocab, d}};
    for (const auto& sh : shapes)
      if (packed_elems(sh[0], sh[1]) * sizeof(uint16_t) >= ((size_t)1 << 31))
        return fail(c, MSD_ERR_INVALID_ARG, "a weight matrix of 2 GiB or more (packed)");
  }
  if (lim->max_batch <= 0 || lim->max_batch > 8 || lim->max_tree <= 0 ||
      lim->max_tree > MSD_MAX_TREE || lim->max_prompt <= 0 || lim->max_seq <= 0 ||
      lim->max_seq % 8)
    return fail(c, MSD_ERR_INVALID_ARG, "bad limits (max_seq must be a multiple of 8)");
  return MSD_OK;
}

struct Up {
  void* dst;
  const void* src;
  size_t bytes;
};

// Copies host arrays to the device through the pinned staging buffer (the
// stream is drained first because the previous upload may still read it).
int upload_many(msd_ctx* c, std::initializer_list<Up> ups) {
  size_t total = 0;
  for (const Up& u : ups) total += (u.bytes + 255) & ~(size_t)255;
  if (total > sizeof(int) * (size_t)STAGE_INTS) return fail(c, MSD_ERR_INVALID_ARG, "upload too large");
  HIPC(c, hipStreamSynchronize(c->st));
  size_t off = 0;
  for (const Up& u : ups) {
    if (!u.bytes) continue;
    char* s = reinterpret_cast<char*>(c->stage) + off;
    std::memcpy(s, u.src, u.bytes);
    HIPC(c, hipMemcpyAsync(u.dst, s, u.bytes, hipMemcpyHostToDevice, c->st));
    off += (u.bytes + 255) & ~(size_t)255;
  }
  return MSD_OK;
}

int upload(msd_ctx* c, int* dst, const int* src, int n) {
  return upload_many(c, {{dst, src, sizeof(int) * (size_t)n}});
}

// The device copy of the call's sequence list; uploaded (which drains the
// stream) only when it differs from the previous call's.
int upload_seqs(msd_ctx* c, const int32_t* seqs, int n) {
  if ((int)c->seq_ids_h.size() == n && std::equal(seqs, seqs + n, c->seq_ids_h.begin()))
    return MSD_OK;
  TRY(upload(c, c->seq_ids, seqs, n));
  c->seq_ids_h.assign(seqs, seqs + n);
  return MSD_OK;
}

// GEMM launch kinds (for the optional trace)
enum { GK_QKV = 0, GK_O = 1, GK_DOWN = 2, GK_GATEUP = 3, GK_FC = 4, GK_LMHEAD = 5 };
constexpr int TK_ATTN = 6;  // trace kind of a tree-attention pass (+ its combine)

// A traced launch of `kind` takes the next pair of the context's events
// (both null when not traced).
void trace_events(msd_ctx* c, int kind, int M, int N, int K, hipEvent_t* e0, hipEvent_t* e1) {
  *e0 = *e1 = nullptr;
  if (!c->tracing || !((c->trace_kinds >> kind) & 1) || c->trace.size() >= c->trace_cap) return;
  msd_ctx::TraceRec r{kind, M, N, K, c->ev_pool[2 * c->trace.size()],
                      c->ev_pool[2 * c->trace.size() + 1]};
  *e0 = r.a;
  *e1 = r.b;
  c->trace.push_back(r);
}

// The caller's row-major matrices of one many-row product (w2: the second
// weight of the SwiGLU pair).
struct RowMajorW {
  const uint16_t *w, *w2;
};

// A many-row product on rocBLAS against row-major bf16 weights: the
// caller's matrices (rm), or else each weight unpacked from the streaming
// layout into a workspace slot (slot w for the pass's weight w; kept for the
// pass's further row chunks, forgotten at the start of every layer pass).
// Then bf16 GEMMs with float32 accumulation and results, issued column-major
// (C^T = W X^T), give the consumer X_hi[m] . W[n] + X_lo[m] . W[n] (at
// column w * off2 + n) in one of two forms:
//  - one product over the 2M rows of K elements that the split rows are
//    (row 2m the hi half of row m, row 2m + 1 its lo half; X's row stride
//    must be 2K): C'[2m + h][n], two partials per row that the consumer
//    sums in hi, lo order;
//  - two products over the strided views X and X + K, the second adding to
//    the first: C[m][n], one partial.
// Either way the sum is hi + lo rounded once.  The one-product form runs
// launches of fewer than BIG_CHUNK rows with results of at most
// BLAS_ONE_PRODUCT_BYTES: its doubled row count tiles better (prefills of
// 640 rows, LLaVA-1.5-7B-shaped, 25.3 -> 20.8 ms; 704 rows, 13B-shaped,
// 46.8 -> 43.2 ms).  Full BIG_CHUNK launches take it for results of at most
// BLAS_ONE_PRODUCT_FULL_BYTES, with the K slices below: 3,136 rows 7B-shaped
// 107.9 -> 100.8 ms, 1,152 rows Qwen2.5-VL-7B-shaped 44.2 -> 37.8 ms.  Their
// SwiGLU pairs (180 and 310 MB of results) keep two products: with the pair
// included, before the K slices, 3,136 rows took 123.4 instead of 111.7 ms.
// A one-product launch with few output tiles is split along K into ns
// slices, one strided batch each (2 ns partials per row: the hi rows of
// every slice, then the lo rows), so that the batches fill the GPU.
#ifndef MAX_K_SLICES
#define MAX_K_SLICES 8
#endif
int blas_gemm(msd_ctx* c, const uint16_t* X, int ldx, int M, const uint16_t* W,
              const uint16_t* W2, int N, int K, int ldp, int off2, const RowMajorW* rm,
              Parts* out) {
  const bool one_product =
      ldx == 2 * K && 2 * (size_t)M * ldp * sizeof(float) <=
                          (M < BIG_CHUNK ? BLAS_ONE_PRODUCT_BYTES : BLAS_ONE_PRODUCT_FULL_BYTES);
  const size_t rows = one_product ? 2 * (size_t)M : (size_t)M;
  if ((!rm && (size_t)N * K > c->plan.wrm_elems) || rows * ldp > c->plan.part_floats)
    return fail(c, MSD_ERR_INVALID_ARG, "internal: prompt GEMM exceeds its buffers");
  // K slices: output tiles counted at 256 x 256; each slice at least 1024
  // columns, a multiple of 8 (16-byte aligned slice starts), within the buffer
  int ns = 1;
  if (one_product) {
    const int tiles = (int)((rows + 255) / 256) * ((N + 255) / 256);
    ns = std::max(1, std::min({MAX_K_SLICES, 256 / std::max(tiles, 1), K / 1024}));
    while (ns > 1 && (K % ns != 0 || (K / ns) % 8 != 0 ||
                      rows * ldp * ns > c->plan.part_floats))
      --ns;
  }
  const int nw = W2 ? 2 : 1, npad = off2;
  const float one = 1.f, zero = 0.f;
  for (int w = 0; w < (W2 ? 2 : 1); ++w) {
    const uint16_t* A = nullptr;
    if (rm) {
      A = w ? rm->w2 : rm->w;
    } else {
      const uint16_t* src = w ? W2 : W;
      uint16_t* wrm = c->wrm + (size_t)w * c->plan.wrm_elems;
      if (c->wrm_src[w] != src) {
        launch_unpack(src, N, K, wrm, c->st);
        LAUNCHED(c);
        c->wrm_src[w] = src;
      }
      A = wrm;
    }
    float* C = c->part + (size_t)w * off2;
    if (ns > 1) {
      // slice s of weight w at column (s nw + w) npad of rows of nw ns npad
      const int ks = K / ns, ldc = nw * ns * npad;
      const rocblas_status st = rocblas_gemm_strided_batched_ex(
          c->blas, rocblas_operation_transpose, rocblas_operation_none, N, (int)rows, ks, &one,
          A, rocblas_datatype_bf16_r, K, ks, X, rocblas_datatype_bf16_r, K, ks, &zero, C,
          rocblas_datatype_f32_r, ldc, (rocblas_stride)nw * npad, C, rocblas_datatype_f32_r, ldc,
          (rocblas_stride)nw * npad, ns, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
      if (st != rocblas_status_success)
        return fail(c, MSD_ERR_HIP,
                    std::string("rocblas_gemm_strided_batched_ex: ") + rocblas_status_to_string(st));
      continue;
    }
    for (int h = 0; h < (one_product ? 1 : 2); ++h) {
      const rocblas_status st = rocblas_gemm_ex(
          c->blas, rocblas_operation_transpose, rocblas_operation_none, N, (int)rows, K, &one, A,
          rocblas_datatype_bf16_r, K, X + (size_t)h * K, rocblas_datatype_bf16_r,
          one_product ? K : ldx, h ? &one : &zero, C, rocblas_datatype_f32_r, ldp, C,
          rocblas_datatype_f32_r, ldp, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
      if (st != rocblas_status_success)
        return fail(c, MSD_ERR_HIP, std::string("rocblas_gemm_ex: ") + rocblas_status_to_string(st));
    }
  }
  if (ns > 1)
    *out = Parts{c->part, 2 * ns, (size_t)nw * npad, 2 * nw * ns * npad, npad};
  else
    *out = one_product ? Parts{c->part, 2, (size_t)ldp, 2 * ldp, off2}
                       : Parts{c->part, 1, (size_t)M * ldp, ldp, off2};
  return MSD_OK;
}

// The target layer's row-major matrices that the prompt products read in
// place.  q, k and v stay unpacked: one product over the stacked q|k|v rows
// keeps more of the GPU busy than three over the caller's separate matrices
// (LLaVA-1.5-7B-shaped 640-row prefill 25.1 ms against 25.9 ms, 3,136 rows
// 109.7 against 114.6 ms).
struct LayerRowMajor {
  RowMajorW o, gu, d;
};
LayerRowMajor layer_row_major(const msd_ctx* c, int l) {
  const LayerW& w = c->layers[l];
  return LayerRowMajor{{w.wo, nullptr}, {w.wg, w.wu}, {w.wd, nullptr}};
}

// Partial products of rows [0, M) of the split rows X (row stride
// ldx = 2K) against the packed weight W [N][K] (and W2); returns the view the
// consumer sums.  Launches of more than CHUNK rows run on rocBLAS, against
// rm's row-major matrices when given.
int gemm(msd_ctx* c, int kind, const uint16_t* X, int ldx, int M, const uint16_t* W,
         const uint16_t* W2, int N, int K, Parts* out, const RowMajorW* rm = nullptr) {
  if (M > CHUNK) {
    if (kind == GK_LMHEAD || M > BIG_CHUNK)
      return fail(c, MSD_ERR_INVALID_ARG, "internal: GEMM launch with too many rows");
    if (!c->blas) return fail(c, MSD_ERR_INVALID_ARG, "internal: many-row GEMM without rocBLAS");
    const int nt = (N + 63) / 64, nw = W2 ? 2 : 1;
    return blas_gemm(c, X, ldx, M, W, W2, N, K, nt * 64 * nw, nt * 64, rm, out);
  }
  const GemmPlan pl = plan_gemm(M, N, K, W2 ? 2 : 1, c->gs.target_wgs);
  if ((size_t)pl.S * M * pl.ldp > c->plan.part_floats)
    return fail(c, MSD_ERR_INVALID_ARG, "internal: GEMM partials exceed their buffer");
  GemmScratch gs = c->gs;
  trace_events(c, kind, M, N, K, &gs.ev_start, &gs.ev_stop);
  launch_gemm(X, ldx, M, W, W2, N, K, c->part, c->sink, gs, c->st);
  LAUNCHED(c);
  *out = Parts{c->part, pl.S, (size_t)M * pl.ldp, pl.ldp, pl.off2};
  return MSD_OK;
}


// Key chunks of a tree-attention pass: each of a workgroup's TREE_WAVES
// waves takes chunk_keys / TREE_WAVES keys (a multiple of 32); enough chunks
// for about ATT_TARGET_WGS workgroups while every wave keeps at least one
// block (a wave hides little latency behind its own blocks, so spreading the
// keys over more CUs pays), at most ATT_MAX_CHUNKS per item (their merge
// reads every chunk's partial at once), within the partial buffer of cap
// floats.
struct TreeChunks {
  int qtiles, chunk_keys, n_chunks;
  size_t part_floats;
};
TreeChunks plan_tree_chunks(const msd_model_desc& m, int n_seq, int nq, int max_ltot,
                            size_t cap) {
  TreeChunks t;
  const int KV = m.n_kv_heads, G = m.n_heads / m.n_kv_heads;
  t.qtiles = (nq * G + 31) / 32;
  const int span = 32 * TREE_WAVES;
  const int base_items = n_seq * KV * t.qtiles;
  const int max_chunks = std::min(ATT_MAX_CHUNKS, std::max(1, (max_ltot + span - 1) / span));
  const int chunks =
      std::min(max_chunks, std::max(1, (ATT_TARGET_WGS + base_items - 1) / base_items));
  int ck = (max_ltot + chunks - 1) / chunks;
  ck = (ck + span - 1) / span * span;
  while ((max_ltot + ck - 1) / ck > ATT_MAX_CHUNKS ||
         attn_partial_floats(n_seq, KV, t.qtiles, (max_ltot + ck - 1) / ck, m.head_dim) > cap)
    ck += span;
  t.chunk_keys = ck;
  t.n_chunks = (max_ltot + ck - 1) / ck;
  t.part_floats = t.n_chunks > 1
                      ? attn_partial_floats(n_seq, KV, t.qtiles, t.n_chunks, m.head_dim)
                      : 0;
  return t;
}

// GEMM input of a normalised layer: xn = x * g (split rows) and the per-row
// sums of squares; the GEMM's consumer applies 1/rms (RMSNorm factored through the
// linear map).
int norm_rows(msd_ctx* c, int rows, const uint16_t* g) {
  launch_resid(Parts{nullptr, 0, 0, 0, 0}, rows, c->m.d_model, RN_KEEP, c->x, g, c->xn, nullptr,
               c->ssq, c->st);
  LAUNCHED(c);
  return MSD_OK;
}

RowNorm row_norm(const msd_ctx* c, int m0) {
  const int nblk = ssq_blocks(c->m.d_model);
  return RowNorm{c->ssq + (size_t)m0 * nblk, nblk, c->m.d_model, c->m.norm_eps};
}

// One decoder stack (the target's layers or the draft's single layer) over
// n_seq * nq rows of c->x described by c->rows; c->xn must hold the first
// layer's input norm.  tree_R < 0 selects causal attention, otherwise tree
// attention over a region of tree_R slots.  After the last layer the rows
// get x += ..., then final_xn = rmsnorm(x) * final_g when final_g and
// final_xb = x when final_xb.
int forward_layers(msd_ctx* c, bool draft, int n_seq, int nq, int tree_R, int max_ltot,
                   const uint16_t* final_g, uint16_t* final_xn, uint16_t* final_xb,
                   const int* feat_dst = nullptr, float* feat = nullptr) {
  const msd_model_desc& m = c->m;
  const int rows = n_seq * nq;
  const int d = m.d_model, H = m.n_heads, KV = m.n_kv_heads, hd = m.head_dim, F = m.ffn_dim;
  const int nl = draft ? 1 : m.n_layers;
  const int ch = row_chunk(rows, tree_R < 0, c->caller_w && !draft && c->blas);
  c->wrm_src[0] = c->wrm_src[1] = nullptr;
  const int B = c->lim.max_batch, S = c->lim.max_seq;
  const size_t layer_kv = (size_t)B * KV * S * hd;
  for (int l = 0; l < nl; ++l) {
    const LayerW& w = draft ? c->dlayer : c->layers[l];
    const PackedLayer& pw = draft ? c->pdlayer : c->players[l];
    const bool rmw = c->caller_w && !draft;
    const LayerRowMajor rl = rmw ? layer_row_major(c, l) : LayerRowMajor{};
    uint16_t* kc = (draft ? c->dk : c->tk) + (size_t)l * layer_kv;
    uint16_t* vc = (draft ? c->dv : c->tv) + (size_t)l * layer_kv;
    Parts pt;
    for (int m0 = 0; m0 < rows; m0 += ch) {
      const int mc = std::min(ch, rows - m0);
      TRY(gemm(c, GK_QKV, c->xn + (size_t)m0 * 2 * d, 2 * d, mc, pw.qkv, nullptr, (H + 2 * KV) * hd,
               d, &pt));
      launch_rope_kv(pt, row_norm(c, m0), mc, H, KV, hd, c->rows.pos + m0, c->rows.seq + m0,
                     c->rows.slot + m0, c->rope, c->q + (size_t)m0 * 2 * H * hd, kc, vc, S, c->st);
      LAUNCHED(c);
    }
    AttnArgs a{};
    a.q = c->q;
    a.kc = kc;
    a.vc = vc;
    for (int i = 0; i < n_seq; ++i) {
      a.seq[i] = c->seq_ids_h[i];
      a.prefix[i] = c->att_pre[i];
      a.keys[i] = c->att_keys[i];
    }
    a.mask = c->rows.mask;
    a.S = S;
    a.H = H;
    a.KV = KV;
    a.hd = hd;
    a.nq = nq;
    a.n_seq = n_seq;
    a.out = c->ao;
    a.scale = 1.0f / std::sqrt((float)hd);
    a.part_o = c->att_po;
    a.part_ml = c->att_ml;
    a.att_cnt = c->att_cnt;
    a.place_err = c->att_place;
    if (tree_R < 0) {
      a.qtiles = (nq + 31) / 32;
      a.n_chunks = 1;
      launch_causal_attention(a, c->st);
    } else {
      const TreeChunks tc = plan_tree_chunks(m, n_seq, nq, max_ltot, c->plan.attn_floats);
      a.qtiles = tc.qtiles;
      a.chunk_keys = tc.chunk_keys;
      a.n_chunks = tc.n_chunks;
      hipEvent_t e0, e1;
      trace_events(c, TK_ATTN, rows, max_ltot, tc.n_chunks, &e0, &e1);
      launch_tree_attention(a, c->st, e0, e1);
    }
    LAUNCHED(c);
    for (int m0 = 0; m0 < rows; m0 += ch) {
      const int mc = std::min(ch, rows - m0);
      TRY(gemm(c, GK_O, c->ao + (size_t)m0 * 2 * H * hd, 2 * H * hd, mc, pw.o, nullptr, d, H * hd,
               &pt, rmw ? &rl.o : nullptr));
      launch_resid(pt, mc, d, RN_ADD, c->x + (size_t)m0 * d, w.n2, c->xn + (size_t)m0 * 2 * d, nullptr,
                   c->ssq + (size_t)m0 * ssq_blocks(d), c->st);
      LAUNCHED(c);
    }
    for (int m0 = 0; m0 < rows; m0 += ch) {
      const int mc = std::min(ch, rows - m0);
      TRY(gemm(c, GK_GATEUP, c->xn + (size_t)m0 * 2 * d, 2 * d, mc, pw.g, pw.u, F, d, &pt,
               rmw ? &rl.gu : nullptr));
      launch_silu(pt, row_norm(c, m0), mc, F, c->act + (size_t)m0 * 2 * F, c->st);
      LAUNCHED(c);
    }
    const bool last = (l + 1 == nl);
    const uint16_t* g_next = last ? final_g : c->layers[l + 1].n1;
    for (int m0 = 0; m0 < rows; m0 += ch) {
      const int mc = std::min(ch, rows - m0);
      TRY(gemm(c, GK_DOWN, c->act + (size_t)m0 * 2 * F, 2 * F, mc, pw.d, nullptr, d, F, &pt,
               rmw ? &rl.d : nullptr));
      if (last && final_g) {
        // the final feature h is materialised (LM head input, draft input)
        launch_resid_norm(pt, 0, mc, d, RN_ADD, c->x + (size_t)m0 * d, final_g, m.norm_eps,
                          final_xn + (size_t)m0 * 2 * d, nullptr, c->st);
      } else {
        launch_resid(pt, mc, d, RN_ADD, c->x + (size_t)m0 * d, last ? nullptr : g_next,
                     last ? nullptr : c->xn + (size_t)m0 * 2 * d,
                     (last && final_xb) ? final_xb + (size_t)m0 * 2 * d : nullptr,
                     last ? nullptr : c->ssq + (size_t)m0 * ssq_blocks(d), c->st,
                     (last && feat) ? feat_dst + m0 : nullptr, last ? feat : nullptr);
      }
      LAUNCHED(c);
    }
  }
  return MSD_OK;
}

// Draft head on rows whose f_down input is in c->fcin (split rows of 2d):
// f = f_down(concat), visual rows replaced by their embeddings, then the
// decoder layer; features in c->x and c->xb, and in the feature slots
// c->rows.dst names (-1: none).
int draft_pass(msd_ctx* c, int n_seq, int nq, int tree_R, int max_ltot, const uint16_t* visual) {
  const int d = c->m.d_model;
  const int rows = n_seq * nq;
  const int ch = row_chunk(rows, tree_R < 0, false);
  Parts pt;
  for (int m0 = 0; m0 < rows; m0 += ch) {
    const int mc = std::min(ch, rows - m0);
    TRY(gemm(c, GK_FC, c->fcin + (size_t)m0 * 4 * d, 4 * d, mc, c->fc_p, nullptr, d, 2 * d, &pt));
    launch_resid(pt, mc, d, RN_SET, c->x + (size_t)m0 * d, visual ? nullptr : c->dlayer.n1,
                 visual ? nullptr : c->xn + (size_t)m0 * 2 * d, nullptr,
                 visual ? nullptr : c->ssq + (size_t)m0 * ssq_blocks(d), c->st);
    LAUNCHED(c);
  }
  if (visual) {
    if (c->visual_input == MSD_DRAFT_VISUAL_FEATURE)
      launch_visual_feature_rows(c->h, c->rows.vis, rows, d, c->x, c->st);
    else
      launch_visual_rows(visual, c->rows.vis, rows, d, c->x, c->st);
    LAUNCHED(c);
    TRY(norm_rows(c, rows, c->dlayer.n1));
  }
  // the final features also go to their draft feature slots (rows.dst)
  return forward_layers(c, true, n_seq, nq, tree_R, max_ltot, nullptr, nullptr, c->xb,
                        c->rows.dst, c->dfeat);
}

// The target over a prompt (or training sequence) of n rows in sequence slot
// seq: row descriptors (the draft's next-token rows included), the slot's
// KV cache rows [0, n) and the final features of every row in c->h.
int prompt_target(msd_ctx* c, int seq, int n, const int32_t* tokens_h,
                  const uint8_t* is_visual_h, const void* visual_d) {
  const int d = c->m.d_model;
  // row descriptors: tok, vis, pos, slot, seq, hrow, dst, nxt
  std::vector<int> a(8 * (size_t)n);
  int* tok = a.data();
  int* vis = tok + n;
  int* pos = vis + n;
  int* slot = pos + n;
  int* sq = slot + n;
  int* hrow = sq + n;
  int* dst = hrow + n;
  int* nxt = dst + n;
  for (int i = 0, v = 0; i < n; ++i) {
    tok[i] = is_visual_h[i] ? 0 : tokens_h[i];
    vis[i] = is_visual_h[i] ? v++ : -1;
    pos[i] = slot[i] = i;
    sq[i] = seq;
    hrow[i] = i;
    dst[i] = (i == n - 1) ? seq * FEAT : -1;
  }
  for (int i = 0; i < n; ++i)
    nxt[i] = (i + 1 < n) ? (is_visual_h[i + 1] ? -1 - vis[i + 1] : tokens_h[i + 1]) : 0;
  int hdr[2] = {0, seq};
  const size_t nb = sizeof(int) * (size_t)n;
  TRY(upload_many(c, {{c->rows.tok, tok, nb}, {c->rows.vis, vis, nb}, {c->rows.pos, pos, nb},
                      {c->rows.slot, slot, nb}, {c->rows.seq, sq, nb}, {c->rows.hrow, hrow, nb},
                      {c->rows.dst, dst, nb}, {c->nxt, nxt, nb}, {c->prefix, hdr, sizeof(int)},
                      {c->seq_ids, hdr + 1, sizeof(int)}}));
  c->seq_ids_h.assign(1, seq);
  c->att_pre[0] = 0;
  c->att_keys[0] = n;
  launch_embed(c->embed, c->rows.tok, c->rows.vis, (const uint16_t*)visual_d, n, d, c->x, c->st);
  LAUNCHED(c);
  TRY(norm_rows(c, n, c->layers[0].n1));
  return forward_layers(c, false, 1, n, -1, n, c->final_norm, c->h, nullptr);
}

// LM head + top-k (and log-sum-exp) over the rows of c->xb: no final norm.
int draft_head(msd_ctx* c, int rows, int k) {
  const int d = c->m.d_model, V = c->m.vocab;
  Parts pt;
  for (int m0 = 0; m0 < rows; m0 += CHUNK) {
    const int mc = std::min(CHUNK, rows - m0);
    TRY(gemm(c, GK_LMHEAD, c->xb + (size_t)m0 * 2 * d, 2 * d, mc, c->lm_p, nullptr, V, d, &pt));
    launch_topk(pt, mc, V, k, c->tk_idx + (size_t)m0 * k, c->tk_val + (size_t)m0 * k,
                c->tk_lse + m0, nullptr, c->tk_scratch, c->st);
    LAUNCHED(c);
  }
  return MSD_OK;
}

int check_seqs(msd_ctx* c, int n_seq, const int32_t* seqs) {
  if (n_seq <= 0 || n_seq > c->lim.max_batch || !seqs)
    return fail(c, MSD_ERR_INVALID_ARG, "bad sequence list");
  for (int i = 0; i < n_seq; ++i) {
    if (seqs[i] < 0 || seqs[i] >= c->lim.max_batch)
      return fail(c, MSD_ERR_INVALID_ARG, "sequence index out of range");
    for (int j = 0; j < i; ++j)
      if (seqs[j] == seqs[i]) return fail(c, MSD_ERR_INVALID_ARG, "duplicate sequence");
    if (!c->ready[seqs[i]]) return fail(c, MSD_ERR_STATE, "sequence has no prompt");
  }
  return MSD_OK;
}

// Validates a static spec and rebuilds the device template when it changes.
int prepare_static(msd_ctx* c, const msd_tree_spec* s) {
  const int N = s->n_nodes, T = N + 1;
  if (!s->parent || !s->rank || N <= 0 || T > c->lim.max_tree)
    return fail(c, MSD_ERR_INVALID_ARG, "bad static tree");
  std::vector<int> par(T, -1), rk(T, 0), dep(T, 0);
  for (int i = 1; i < T; ++i) {
    par[i] = s->parent[i - 1];
    rk[i] = s->rank[i - 1];
    if (par[i] < 0 || par[i] >= i) return fail(c, MSD_ERR_INVALID_ARG, "parent must precede child");
    if (rk[i] < 0 || rk[i] >= TOPK) return fail(c, MSD_ERR_INVALID_ARG, "rank out of range");
    dep[i] = dep[par[i]] + 1;
    if (dep[i] < dep[i - 1]) return fail(c, MSD_ERR_INVALID_ARG, "nodes not ordered by depth");
    for (int j = 1; j < i; ++j)
      if (par[j] == par[i] && rk[j] == rk[i])
        return fail(c, MSD_ERR_INVALID_ARG, "siblings share a rank");
  }
  if (T == c->sp_T && par == c->sp_parent && rk == c->sp_rank) return MSD_OK;
  const int D = dep[T - 1];
  std::vector<int> has(T, 0);
  for (int i = 1; i < T; ++i) has[par[i]] = 1;
  std::vector<int> exp_idx(T, -1), pslot(T, 0), rnodes, rpos(T, 0);
  std::vector<uint64_t> anc(T, 0), emask(T, 0);
  c->round_off.assign(D, 0);
  c->round_n.assign(D, 0);
  c->round_k.assign(D, 0);
  c->round_exp_end.assign(D, 0);
  int ne = 0;
  for (int dd = 0; dd < D; ++dd) {
    c->round_off[dd] = (int)rnodes.size();
    for (int u = 0; u < T; ++u) {
      if (dep[u] != dd || !has[u]) continue;
      rpos[u] = c->round_n[dd]++;
      if (dd > 0) {
        rnodes.push_back(u);
        exp_idx[u] = ne++;
      }
    }
    if (dd == 0) c->round_n[dd] = 1;
    c->round_exp_end[dd] = ne;
  }
  for (int i = 0; i < T; ++i) {
    anc[i] = (i ? anc[par[i]] : 0ull) | (1ull << i);
    if (i > 0) {
      const int p = par[i];
      pslot[i] = (p == 0) ? 0 : 1 + exp_idx[p];
      c->round_k[dep[p]] = std::max(c->round_k[dep[p]], rk[i] + 1);
    }
    if (exp_idx[i] >= 0) emask[i] = (par[i] > 0 ? emask[par[i]] : 0ull) | (1ull << exp_idx[i]);
  }
  if (ne > MSD_MAX_TREE) return fail(c, MSD_ERR_INVALID_ARG, "too many expanded nodes");
  rnodes.resize(MSD_MAX_TREE, 0);
  std::vector<int> packed;
  auto put = [&](const std::vector<int>& v) { packed.insert(packed.end(), v.begin(), v.end()); packed.resize(packed.size() + (MSD_MAX_TREE - v.size()), 0); };
  put(par); put(rk); put(dep); put(exp_idx); put(pslot); put(rnodes); put(rpos);
  std::vector<int> anc_i(2 * MSD_MAX_TREE, 0), em_i(2 * MSD_MAX_TREE, 0);
  std::memcpy(anc_i.data(), anc.data(), sizeof(uint64_t) * T);
  std::memcpy(em_i.data(), emask.data(), sizeof(uint64_t) * T);
  TRY(upload(c, c->sp.parent, packed.data(), MSD_MAX_TREE));
  TRY(upload(c, c->sp.rank, packed.data() + MSD_MAX_TREE, MSD_MAX_TREE));
  TRY(upload(c, c->sp.depth, packed.data() + 2 * MSD_MAX_TREE, MSD_MAX_TREE));
  TRY(upload(c, c->sp.exp_idx, packed.data() + 3 * MSD_MAX_TREE, MSD_MAX_TREE));
  TRY(upload(c, c->sp.pslot, packed.data() + 4 * MSD_MAX_TREE, MSD_MAX_TREE));
  TRY(upload(c, c->sp.round_nodes, packed.data() + 5 * MSD_MAX_TREE, MSD_MAX_TREE));
  TRY(upload(c, c->sp.round_pos, packed.data() + 6 * MSD_MAX_TREE, MSD_MAX_TREE));
  TRY(upload(c, (int*)c->sp.anc, anc_i.data(), 2 * MSD_MAX_TREE));
  TRY(upload(c, (int*)c->sp.exp_mask, em_i.data(), 2 * MSD_MAX_TREE));
  c->sp_T = T;
  c->sp_D = D;
  c->sp_parent = par;
  c->sp_rank = rk;
  return MSD_OK;
}

// Checks shared by the two acceptance calls.
int check_accept(msd_ctx* c, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d,
                 int n_nodes, int32_t* emitted_h, int32_t* n_emitted_h) {
  TRY(check_seqs(c, n_seq, seqs_h));
  if (!trees_d || !emitted_h || !n_emitted_h) return fail(c, MSD_ERR_INVALID_ARG, "null argument");
  if (c->verified_T == 0 || n_nodes != c->verified_T ||
      !std::equal(seqs_h, seqs_h + n_seq, c->verified_seqs.begin(), c->verified_seqs.end()))
    return fail(c, MSD_ERR_STATE, "accept must follow msd_verify of the same sequences and trees");
  return upload_seqs(c, seqs_h, n_seq);
}

// After the accepted paths are in acc_path / acc_n / acc_emit: compaction of
// the target cache, the pending draft rows, and the host copy of the
// emitted tokens (the one wait of the cycle).
int finish_accept(msd_ctx* c, int n_seq, const int32_t* seqs_h, int T, int32_t* emitted_h,
                  int32_t* n_emitted_h) {
  const int d = c->m.d_model;
  launch_compact(c->tk, c->tv, c->m.n_layers, c->lim.max_batch, c->m.n_kv_heads, c->lim.max_seq,
                 c->m.head_dim, n_seq, c->seq_ids, c->acc_path, c->acc_n, c->d_len, c->st);
  LAUNCHED(c);
  launch_commit(n_seq, c->seq_ids, c->acc_path, c->acc_n, c->acc_emit, c->h, T, d, c->pend_h,
                c->pend_next, c->pend_n, PEND, c->d_len, c->d_root, c->st);
  LAUNCHED(c);
  // the staging block's last 64 ints take other small read-backs
  static_assert(ACC_BACK_INTS <= 544, "acceptance read-back block");
  int* back = c->stage + STAGE_INTS - 64 - 544;
  HIPC(c, hipMemcpyAsync(back, c->acc_emit, sizeof(int) * ACC_BACK_INTS, hipMemcpyDeviceToHost,
                         c->st));
  HIPC(c, hipStreamSynchronize(c->st));
  c->verified_T = 0;
  if (back[MSD_MAX_TREE * 8 + 16]) {
    HIPC(c, hipMemsetAsync(c->att_place, 0, sizeof(int), c->st));
    HIPC(c, hipStreamSynchronize(c->st));
    return fail(c, MSD_ERR_HIP,
                "tree attention found the key chunks of one item on different XCDs (the "
                "workgroup placement its in-L2 merge relies on); results since the last "
                "acceptance are unreliable");
  }
  for (int i = 0; i < n_seq; ++i)
    if (back[MSD_MAX_TREE * 8 + 8 + i]) {
      // the kernels accepted nothing for any sequence of the call
      for (int k = 0; k < n_seq; ++k) n_emitted_h[k] = 0;
      return fail(c, MSD_ERR_INVALID_ARG,
                  "malformed tree for call slot " + std::to_string(i) +
                      " (parent order, depth, ancestor mask, token id or duplicate sibling); "
                      "nothing was accepted");
    }
  for (int i = 0; i < n_seq; ++i) {
    const int n = back[MSD_MAX_TREE * 8 + i];
    n_emitted_h[i] = n;
    for (int j = 0; j < MSD_MAX_TREE; ++j) emitted_h[i * MSD_MAX_TREE + j] = back[i * MSD_MAX_TREE + j];
    c->L[seqs_h[i]] += n;
    c->pend[seqs_h[i]] = n;
  }
  return MSD_OK;
}

// ------------------------------------------------------------------------
// Draft-head training (Sec. 4.2; the state is TrainState).
void train_free(TrainState* t) {
  if (!t) return;
  for (void* p : t->allocs) (void)hipFree(p);
  if (t->blas) (void)rocblas_destroy_handle(t->blas);
  delete t;
}

// Row-major C[M][N] = alpha op(A) op(B) + beta C (ta: A stored [K][M];
// tb: B stored [N][K]); rocBLAS is column-major, so it computes the
// transposed product C^T = op(B)^T op(A)^T.
int sgemm_rm(msd_ctx* c, bool ta, bool tb, int M, int N, int K, float alpha, const float* A,
             int lda, const float* B, int ldb, float beta, float* C, int ldc) {
  const rocblas_status st = rocblas_sgemm(
      c->tr->blas, tb ? rocblas_operation_transpose : rocblas_operation_none,
      ta ? rocblas_operation_transpose : rocblas_operation_none, N, M, K, &alpha, B, ldb, A, lda,
      &beta, C, ldc);
  if (st != rocblas_status_success)
    return fail(c, MSD_ERR_HIP, std::string("rocblas_sgemm: ") + rocblas_status_to_string(st));
  return MSD_OK;
}

// Shapes [rows][cols] of the draft parameters in training order.
void train_shapes(const msd_model_desc& m, int (*sh)[2]) {
  const int d = m.d_model, F = m.ffn_dim, qd = m.n_heads * m.head_dim;
  const int kd = m.n_kv_heads * m.head_dim;
  const int s[TRAIN_PARAMS][2] = {{d, 2 * d}, {qd, d}, {kd, d}, {kd, d}, {d, qd},
                                  {F, d},     {F, d},  {d, F},  {1, d},  {1, d}};
  for (int i = 0; i < TRAIN_PARAMS; ++i) sh[i][0] = s[i][0], sh[i][1] = s[i][1];
}

int train_init(msd_ctx* c) {
  if (c->tr) return MSD_OK;
  const msd_model_desc& m = c->m;
  const int d = m.d_model, F = m.ffn_dim, H = m.n_heads, KV = m.n_kv_heads, hd = m.head_dim;
  const int V = m.vocab, R = c->lim.max_prompt - 1;
  TrainState* t = new TrainState;
  t->Rmax = R;
  int sh[TRAIN_PARAMS][2];
  train_shapes(m, sh);
  for (int i = 0; i < TRAIN_PARAMS; ++i) t->off[i + 1] = t->off[i] + (size_t)sh[i][0] * sh[i][1];
  const size_t np = t->off[TRAIN_PARAMS];
  auto take = [&](size_t bytes) -> void* {
    void* p = nullptr;
    if (hipMalloc(&p, std::max<size_t>(bytes, 256)) != hipSuccess) return nullptr;
    t->allocs.push_back(p);
    return p;
  };
  auto f32 = [&](size_t n) { return static_cast<float*>(take(n * sizeof(float))); };
  t->w = f32(np);
  t->g = f32(np);
  t->m = f32(np);
  t->v = f32(np);
  t->wb = static_cast<uint16_t*>(take(np * sizeof(uint16_t)));
  t->lm = f32((size_t)V * d);
  const size_t Rd = (size_t)R * d, RF = (size_t)R * F, RV = (size_t)R * V;
  t->H = f32((size_t)(R + 1) * d);
  t->X0 = f32(2 * Rd);
  t->E0 = f32(Rd);
  t->F = f32(Rd);
  t->A1 = f32(Rd);
  t->r1 = f32(R);
  t->Q = f32((size_t)R * H * hd);
  t->K = f32((size_t)R * KV * hd);
  t->V = f32((size_t)R * KV * hd);
  t->S = f32((size_t)H * R * R);
  t->dP = f32((size_t)H * R * R);
  t->O = f32((size_t)R * H * hd);
  t->X1 = f32(Rd);
  t->A2 = f32(Rd);
  t->r2 = f32(R);
  t->G = f32(RF);
  t->U = f32(RF);
  t->Mx = f32(RF);
  t->D = f32(Rd);
  t->Ld = f32(RV);
  t->Lt = f32(RV);
  t->dD = f32(Rd);
  t->dMx = f32(RF);
  t->dG = f32(RF);
  t->dU = f32(RF);
  t->dA2 = f32(Rd);
  t->dX1 = f32(Rd);
  t->dO = f32((size_t)R * H * hd);
  t->dQ = f32((size_t)R * H * hd);
  t->dK = f32((size_t)R * KV * hd);
  t->dV = f32((size_t)R * KV * hd);
  t->dA1 = f32(Rd);
  t->dF = f32(Rd);
  t->reg = f32(R);
  t->ce = f32(R);
  for (void* p : t->allocs)
    if (!p) {
      train_free(t);
      return fail(c, MSD_ERR_HIP, "training buffers: hipMalloc failed");
    }
  if (rocblas_create_handle(&t->blas) != rocblas_status_success ||
      rocblas_set_stream(t->blas, c->st) != rocblas_status_success) {
    train_free(t);
    return fail(c, MSD_ERR_HIP, "rocblas handle");
  }
  c->tr = t;
  // the draft's parameters from the packed copies the decoder uses (and the
  // norm gains); from here on the decoder reads the gains from wb
  const PackedLayer& pl = c->pdlayer;
  const size_t pq = packed_elems(H * hd, d), pk = packed_elems(KV * hd, d);
  const uint16_t* packed[7] = {c->fc_p, pl.qkv, pl.qkv + pq, pl.qkv + pq + pk, pl.o, pl.g, pl.u};
  for (int i = 0; i < 7; ++i) launch_unpack(packed[i], sh[i][0], sh[i][1], t->wb + t->off[i], c->st);
  launch_unpack(pl.d, sh[7][0], sh[7][1], t->wb + t->off[7], c->st);
  HIPC(c, hipMemcpyAsync(t->wb + t->off[8], c->dlayer.n1, sizeof(uint16_t) * d,
                         hipMemcpyDeviceToDevice, c->st));
  HIPC(c, hipMemcpyAsync(t->wb + t->off[9], c->dlayer.n2, sizeof(uint16_t) * d,
                         hipMemcpyDeviceToDevice, c->st));
  LAUNCHED(c);
  tr_widen(t->wb, np, t->w, c->st);
  tr_fill(t->g, np, 0.f, c->st);
  tr_fill(t->m, np, 0.f, c->st);
  tr_fill(t->v, np, 0.f, c->st);
  uint16_t* lm16 = static_cast<uint16_t*>(take((size_t)V * d * sizeof(uint16_t)));
  if (!lm16) return fail(c, MSD_ERR_HIP, "training buffers: hipMalloc failed");
  launch_unpack(c->lm_p, V, d, lm16, c->st);
  tr_widen(lm16, (size_t)V * d, t->lm, c->st);
  LAUNCHED(c);
  c->dlayer.n1 = t->wb + t->off[8];
  c->dlayer.n2 = t->wb + t->off[9];
  HIPC(c, hipStreamSynchronize(c->st));
  return MSD_OK;
}

// One training sequence: forward, loss and gradient sums (see
// msd_train_accumulate).  c->h holds the target features of its n rows,
// c->rows.tok / .vis its tokens and visual row indices.
int train_pass(msd_ctx* c, int n, const void* visual_d, double* loss3) {
  TrainState* t = c->tr;
  const msd_model_desc& m = c->m;
  const int d = m.d_model, F = m.ffn_dim, H = m.n_heads, KV = m.n_kv_heads, hd = m.head_dim;
  const int V = m.vocab, R = n - 1, Gq = H / KV, qd = H * hd, kd = KV * hd;
  const float eps = m.norm_eps, scale = 1.f / std::sqrt((float)hd);
  hipStream_t st = c->st;
  const size_t* o = t->off;
  float* w = t->w;
  float* g = t->g;
  const float *Wfc = w + o[0], *Wq = w + o[1], *Wk = w + o[2], *Wv = w + o[3], *Wo = w + o[4];
  const float *Wg = w + o[5], *Wu = w + o[6], *Wd = w + o[7], *n1 = w + o[8], *n2 = w + o[9];
  const size_t Rd = (size_t)R * d;
  // ---- forward
  tr_inputs(c->h, c->embed, c->rows.tok, c->rows.vis, (const uint16_t*)visual_d, n, d,
            c->visual_input == MSD_DRAFT_VISUAL_FEATURE, t->H, t->X0, t->E0, st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, false, true, R, d, 2 * d, 1.f, t->X0, 2 * d, Wfc, 2 * d, 0.f, t->F, d));
  tr_visual_rows(t->F, t->E0, c->rows.vis, R, d, st);
  tr_rmsnorm(t->F, n1, eps, R, d, t->A1, t->r1, st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, false, true, R, qd, d, 1.f, t->A1, d, Wq, d, 0.f, t->Q, qd));
  TRY(sgemm_rm(c, false, true, R, kd, d, 1.f, t->A1, d, Wk, d, 0.f, t->K, kd));
  TRY(sgemm_rm(c, false, true, R, kd, d, 1.f, t->A1, d, Wv, d, 0.f, t->V, kd));
  tr_rope(t->Q, R, H, hd, c->rope, 1, st);
  tr_rope(t->K, R, KV, hd, c->rope, 1, st);
  LAUNCHED(c);
  const size_t RR = (size_t)R * R;
  for (int h = 0; h < H; ++h)
    TRY(sgemm_rm(c, false, true, R, R, hd, 1.f, t->Q + h * hd, qd, t->K + (h / Gq) * hd, kd, 0.f,
                 t->S + h * RR, R));
  tr_softmax(t->S, R, H, scale, st);
  LAUNCHED(c);
  for (int h = 0; h < H; ++h)
    TRY(sgemm_rm(c, false, false, R, hd, R, 1.f, t->S + h * RR, R, t->V + (h / Gq) * hd, kd, 0.f,
                 t->O + h * hd, qd));
  HIPC(c, hipMemcpyAsync(t->X1, t->F, Rd * 4, hipMemcpyDeviceToDevice, st));
  TRY(sgemm_rm(c, false, true, R, d, qd, 1.f, t->O, qd, Wo, qd, 1.f, t->X1, d));
  tr_rmsnorm(t->X1, n2, eps, R, d, t->A2, t->r2, st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, false, true, R, F, d, 1.f, t->A2, d, Wg, d, 0.f, t->G, F));
  TRY(sgemm_rm(c, false, true, R, F, d, 1.f, t->A2, d, Wu, d, 0.f, t->U, F));
  tr_silu(t->G, t->U, (size_t)R * F, t->Mx, st);
  LAUNCHED(c);
  HIPC(c, hipMemcpyAsync(t->D, t->X1, Rd * 4, hipMemcpyDeviceToDevice, st));
  TRY(sgemm_rm(c, false, true, R, d, F, 1.f, t->Mx, F, Wd, F, 1.f, t->D, d));
  // ---- loss: regression toward h_{i+1}, token term against softmax(W_lm h_{i+1})
  tr_reg(t->D, t->H, R, d, t->dD, t->reg, st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, false, true, R, V, d, 1.f, t->D, d, t->lm, d, 0.f, t->Ld, V));
  TRY(sgemm_rm(c, false, true, R, V, d, 1.f, t->H + d, d, t->lm, d, 0.f, t->Lt, V));
  tr_ce(t->Ld, t->Lt, R, V, TRAIN_CLS_WEIGHT, t->ce, st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, false, false, R, d, V, 1.f, t->Ld, V, t->lm, d, 1.f, t->dD, d));
  // ---- backward (gradient sums over the rows, accumulated into g)
  TRY(sgemm_rm(c, true, false, d, F, R, 1.f, t->dD, d, t->Mx, F, 1.f, g + o[7], F));
  TRY(sgemm_rm(c, false, false, R, F, d, 1.f, t->dD, d, Wd, F, 0.f, t->dMx, F));
  tr_silu_bwd(t->G, t->U, t->dMx, (size_t)R * F, t->dG, t->dU, st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, true, false, F, d, R, 1.f, t->dG, F, t->A2, d, 1.f, g + o[5], d));
  TRY(sgemm_rm(c, true, false, F, d, R, 1.f, t->dU, F, t->A2, d, 1.f, g + o[6], d));
  TRY(sgemm_rm(c, false, false, R, d, F, 1.f, t->dG, F, Wg, d, 0.f, t->dA2, d));
  TRY(sgemm_rm(c, false, false, R, d, F, 1.f, t->dU, F, Wu, d, 1.f, t->dA2, d));
  HIPC(c, hipMemcpyAsync(t->dX1, t->dD, Rd * 4, hipMemcpyDeviceToDevice, st));
  tr_rmsnorm_bwd(t->X1, n2, t->r2, t->dA2, R, d, t->dX1, g + o[9], st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, true, false, d, qd, R, 1.f, t->dX1, d, t->O, qd, 1.f, g + o[4], qd));
  TRY(sgemm_rm(c, false, false, R, qd, d, 1.f, t->dX1, d, Wo, qd, 0.f, t->dO, qd));
  tr_fill(t->dK, (size_t)R * kd, 0.f, st);
  tr_fill(t->dV, (size_t)R * kd, 0.f, st);
  LAUNCHED(c);
  for (int h = 0; h < H; ++h) {
    const int kv = h / Gq;
    TRY(sgemm_rm(c, true, false, R, hd, R, 1.f, t->S + h * RR, R, t->dO + h * hd, qd, 1.f,
                 t->dV + kv * hd, kd));
    TRY(sgemm_rm(c, false, true, R, R, hd, 1.f, t->dO + h * hd, qd, t->V + kv * hd, kd, 0.f,
                 t->dP + h * RR, R));
  }
  tr_softmax_bwd(t->S, t->dP, R, H, scale, st);
  LAUNCHED(c);
  for (int h = 0; h < H; ++h) {
    const int kv = h / Gq;
    TRY(sgemm_rm(c, false, false, R, hd, R, 1.f, t->dP + h * RR, R, t->K + kv * hd, kd, 0.f,
                 t->dQ + h * hd, qd));
    TRY(sgemm_rm(c, true, false, R, hd, R, 1.f, t->dP + h * RR, R, t->Q + h * hd, qd, 1.f,
                 t->dK + kv * hd, kd));
  }
  tr_rope(t->dQ, R, H, hd, c->rope, -1, st);
  tr_rope(t->dK, R, KV, hd, c->rope, -1, st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, true, false, qd, d, R, 1.f, t->dQ, qd, t->A1, d, 1.f, g + o[1], d));
  TRY(sgemm_rm(c, true, false, kd, d, R, 1.f, t->dK, kd, t->A1, d, 1.f, g + o[2], d));
  TRY(sgemm_rm(c, true, false, kd, d, R, 1.f, t->dV, kd, t->A1, d, 1.f, g + o[3], d));
  TRY(sgemm_rm(c, false, false, R, d, qd, 1.f, t->dQ, qd, Wq, d, 0.f, t->dA1, d));
  TRY(sgemm_rm(c, false, false, R, d, kd, 1.f, t->dK, kd, Wk, d, 1.f, t->dA1, d));
  TRY(sgemm_rm(c, false, false, R, d, kd, 1.f, t->dV, kd, Wv, d, 1.f, t->dA1, d));
  HIPC(c, hipMemcpyAsync(t->dF, t->dX1, Rd * 4, hipMemcpyDeviceToDevice, st));
  tr_rmsnorm_bwd(t->F, n1, t->r1, t->dA1, R, d, t->dF, g + o[8], st);
  tr_zero_visual(t->dF, c->rows.vis, R, d, st);
  LAUNCHED(c);
  TRY(sgemm_rm(c, true, false, d, 2 * d, R, 1.f, t->dF, d, t->X0, 2 * d, 1.f, g + o[0], 2 * d));
  // the rows' loss terms, summed in row order on the host
  std::vector<float> rc(2 * (size_t)R);
  HIPC(c, hipMemcpyAsync(rc.data(), t->reg, sizeof(float) * R, hipMemcpyDeviceToHost, st));
  HIPC(c, hipMemcpyAsync(rc.data() + R, t->ce, sizeof(float) * R, hipMemcpyDeviceToHost, st));
  HIPC(c, hipStreamSynchronize(st));
  double reg = 0, ce = 0;
  for (int i = 0; i < R; ++i) {
    reg += rc[i];
    ce += rc[R + i];
  }
  loss3[0] = reg + TRAIN_CLS_WEIGHT * ce;
  loss3[1] = reg;
  loss3[2] = ce;
  t->rows += R;
  return MSD_OK;
}

// rocBLAS loads the kernels of a GEMM shape on its first use (about 0.2 s
// for a context's first prompt).  Run once here, on layer 0's weights and
// whatever the activation buffers hold, each prompt GEMM shape at the row
// counts this context's prompts will use: full BIG_CHUNK launches and the
// launch of a max_prompt-row prompt's last chunk.  The results are
// discarded.
int warm_blas(msd_ctx* c) {
  if (!c->blas) return MSD_OK;
  const msd_model_desc& m = c->m;
  const int d = m.d_model, F = m.ffn_dim, hh = m.n_heads * m.head_dim;
  const int rows = c->lim.max_prompt;
  std::vector<int> ms;
  if (rows >= BIG_CHUNK) ms.push_back(BIG_CHUNK);
  const int tail = rows % BIG_CHUNK;
  if (rows > PROMPT_BIG_MIN_ROWS && tail > CHUNK) ms.push_back(tail);
  const PackedLayer& p = c->players[0];
  for (int M : ms) {
    Parts pt;
    TRY(gemm(c, GK_QKV, c->xn, 2 * d, M, p.qkv, nullptr, c->plan.ld_qkv, d, &pt));
    TRY(gemm(c, GK_O, c->ao, 2 * hh, M, p.o, nullptr, d, hh, &pt));
    TRY(gemm(c, GK_GATEUP, c->xn, 2 * d, M, p.g, p.u, F, d, &pt));
    TRY(gemm(c, GK_DOWN, c->act, 2 * F, M, p.d, nullptr, d, F, &pt));
    TRY(gemm(c, GK_FC, c->fcin, 4 * d, M, c->fc_p, nullptr, d, 2 * d, &pt));
  }
  c->wrm_src[0] = c->wrm_src[1] = nullptr;
  HIPC(c, hipStreamSynchronize(c->st));
  return MSD_OK;
}

}  // namespace

extern "C" {

int msd_buffer_sizes(const msd_model_desc* m, const msd_limits* lim, size_t* target_kv_bytes,
                     size_t* draft_kv_bytes, size_t* workspace_bytes, size_t* weight_bytes) {
  int r = check_desc(m, lim, nullptr);
  if (r != MSD_OK) return r;
  if (target_kv_bytes) *target_kv_bytes = kv_bytes(*m, *lim, m->n_layers);
  if (draft_kv_bytes) *draft_kv_bytes = kv_bytes(*m, *lim, 1);
  if (workspace_bytes) *workspace_bytes = carve(nullptr, *m, *lim, nullptr);
  if (weight_bytes) *weight_bytes = weight_layout(*m).total * sizeof(uint16_t);
  return MSD_OK;
}

int msd_workspace_size(const msd_model_desc* m, const msd_limits* lim, size_t* bytes) {
  if (!bytes) return fail(nullptr, MSD_ERR_INVALID_ARG, "null output pointer");
  return msd_buffer_sizes(m, lim, nullptr, nullptr, bytes, nullptr);
}

int msd_create(const msd_model_desc* m, const msd_limits* lim, const msd_target_weights* tw,
               const msd_draft_weights* dw, const msd_buffers* bufs, void* stream,
               msd_ctx** out) {
  if (!out) return fail(nullptr, MSD_ERR_INVALID_ARG, "null output pointer");
  *out = nullptr;
  int r = check_desc(m, lim, nullptr);
  if (r != MSD_OK) return r;
  if (!tw || !dw || !bufs || !tw->embed || !tw->layers || !tw->final_norm || !tw->lm_head ||
      !dw->fc || !bufs->target_k || !bufs->target_v || !bufs->draft_k || !bufs->draft_v ||
      !bufs->workspace || !bufs->packed_weights)
    return fail(nullptr, MSD_ERR_INVALID_ARG, "null weight or buffer pointer");
  for (int l = 0; l <= m->n_layers; ++l) {
    const msd_layer_weights& w = l < m->n_layers ? tw->layers[l] : dw->layer;
    if (!w.wq || !w.wk || !w.wv || !w.wo || !w.w_gate || !w.w_up || !w.w_down || !w.attn_norm ||
        !w.ffn_norm)
      return fail(nullptr, MSD_ERR_INVALID_ARG, "null layer weight");
  }
  msd_ctx* c = new msd_ctx();
  c->m = *m;
  c->lim = *lim;
  c->plan = make_plan(*m, *lim);
  c->st = (hipStream_t)stream;
  for (int l = 0; l < m->n_layers; ++l) c->layers.push_back(to_layer(tw->layers[l]));
  c->dlayer = to_layer(dw->layer);
  c->embed = (const uint16_t*)tw->embed;
  c->final_norm = (const uint16_t*)tw->final_norm;
  // packed copies of every GEMM weight in the caller's arena
  const WeightLayout wl = weight_layout(*m);
  uint16_t* arena = (uint16_t*)bufs->packed_weights;
  for (int l = 0; l <= m->n_layers; ++l) {
    uint16_t* b = arena + wl.layer_off[l];
    const PackedLayer pl{b, b + wl.qkv, b + wl.qkv + wl.o, b + wl.qkv + wl.o + wl.g,
                         b + wl.qkv + wl.o + wl.g + wl.u};
    if (l < m->n_layers) c->players.push_back(pl);
    else c->pdlayer = pl;
  }
  c->fc_p = arena + wl.fc_off;
  c->lm_p = arena + wl.lm_off;
  c->tk = (uint16_t*)bufs->target_k;
  c->tv = (uint16_t*)bufs->target_v;
  c->dk = (uint16_t*)bufs->draft_k;
  c->dv = (uint16_t*)bufs->draft_v;
  carve(c, *m, *lim, (char*)bufs->workspace);
  if (c->plan.wrm_elems) {
    // prompt GEMMs on rocBLAS, on the context's stream, in a workspace carved
    // from the caller's buffer (the context's destructor frees the handle)
    rocblas_handle hb = nullptr;
    const bool ok = rocblas_create_handle(&hb) == rocblas_status_success;
    if (ok) c->blas = hb;
    if (!ok || rocblas_set_stream(c->blas, c->st) != rocblas_status_success ||
        rocblas_set_workspace(c->blas, c->blas_ws, BLAS_WS_BYTES) != rocblas_status_success) {
      delete c;
      return fail(nullptr, MSD_ERR_HIP, "rocBLAS handle for the prompt GEMMs");
    }
  }
  {
    hipError_t e = hipGetDevice(&c->device);
    void* sp = nullptr;
    if (e == hipSuccess) e = noalloc_scratch(c->device, &sp);
    if (e != hipSuccess) {
      delete c;
      return fail(nullptr, MSD_ERR_HIP,
                  std::string("resolving the no-allocation scratch: ") + hipGetErrorString(e));
    }
    c->noalloc_base = static_cast<float*>(sp);
  }
  c->gs.target_wgs = GEMM_WGS;
  c->gs.ev_start = nullptr;
  c->gs.ev_stop = nullptr;
  c->L.assign(lim->max_batch, 0);
  c->pend.assign(lim->max_batch, 0);
  c->ready.assign(lim->max_batch, 0);
  hipError_t e = hipHostMalloc((void**)&c->stage, sizeof(int) * STAGE_INTS, hipHostMallocDefault);
  if (e != hipSuccess) {
    delete c;
    return fail(nullptr, MSD_ERR_HIP, std::string("hipHostMalloc: ") + hipGetErrorString(e));
  }
  auto init = [&]() -> int {
    // never-written cache slots may be read (with zero weight) by padded rows
    const size_t tkv = kv_bytes(*m, *lim, m->n_layers), dkv = kv_bytes(*m, *lim, 1);
    HIPC(c, hipMemsetAsync(c->tk, 0, tkv, c->st));
    HIPC(c, hipMemsetAsync(c->tv, 0, tkv, c->st));
    HIPC(c, hipMemsetAsync(c->dk, 0, dkv, c->st));
    HIPC(c, hipMemsetAsync(c->dv, 0, dkv, c->st));
    HIPC(c, hipMemsetAsync(c->d_len, 0, sizeof(int) * lim->max_batch, c->st));
    HIPC(c, hipMemsetAsync(c->pend_n, 0, sizeof(int) * lim->max_batch, c->st));
    HIPC(c, hipMemsetAsync(c->d_root, 0, sizeof(int) * lim->max_batch, c->st));
    HIPC(c, hipMemsetAsync(c->tree_err, 0, sizeof(int) * lim->max_batch, c->st));
    HIPC(c, hipMemsetAsync(c->att_cnt, 0, sizeof(int) * c->plan.att_items, c->st));
    HIPC(c, hipMemsetAsync(c->att_place, 0, sizeof(int), c->st));
    launch_rope_table(c->rope, lim->max_seq, m->head_dim, (double)m->rope_theta, c->st);
    LAUNCHED(c);
    const int d = m->d_model, hd = m->head_dim, H = m->n_heads, KV = m->n_kv_heads;
    const int F = m->ffn_dim;
    for (int l = 0; l <= m->n_layers; ++l) {
      const LayerW& w = l < m->n_layers ? c->layers[l] : c->dlayer;
      const PackedLayer& p = l < m->n_layers ? c->players[l] : c->pdlayer;
      uint16_t* qkv = const_cast<uint16_t*>(p.qkv);
      launch_pack(w.wq, H * hd, d, qkv, c->st);
      launch_pack(w.wk, KV * hd, d, qkv + packed_elems(H * hd, d), c->st);
      launch_pack(w.wv, KV * hd, d, qkv + packed_elems(H * hd, d) + packed_elems(KV * hd, d), c->st);
      launch_pack(w.wo, d, H * hd, const_cast<uint16_t*>(p.o), c->st);
      launch_pack(w.wg, F, d, const_cast<uint16_t*>(p.g), c->st);
      launch_pack(w.wu, F, d, const_cast<uint16_t*>(p.u), c->st);
      launch_pack(w.wd, d, F, const_cast<uint16_t*>(p.d), c->st);
      LAUNCHED(c);
    }
    launch_pack((const uint16_t*)dw->fc, d, 2 * d, const_cast<uint16_t*>(c->fc_p), c->st);
    launch_pack((const uint16_t*)tw->lm_head, m->vocab, d, const_cast<uint16_t*>(c->lm_p), c->st);
    LAUNCHED(c);
    HIPC(c, hipStreamSynchronize(c->st));
    return MSD_OK;
  };
  r = init();
  if (r == MSD_OK) r = warm_blas(c);
  if (r != MSD_OK) {
    g_err = c->err;
    (void)hipHostFree(c->stage);
    delete c;
    return r;
  }
  *out = c;
  return MSD_OK;
}

int msd_destroy(msd_ctx* c) {
  if (!c) return MSD_OK;
  const hipError_t e1 = hipStreamSynchronize(c->st);
  train_free(c->tr);
  for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
  const hipError_t e2 = hipHostFree(c->stage);
  delete c;
  if (e1 != hipSuccess || e2 != hipSuccess) {
    g_err = std::string("msd_destroy: ") + hipGetErrorString(e1 != hipSuccess ? e1 : e2);
    return MSD_ERR_HIP;
  }
  return MSD_OK;
}

const char* msd_last_error(const msd_ctx* c) { return c ? c->err.c_str() : g_err.c_str(); }

int msd_seq_len(const msd_ctx* c, int seq) {
  if (!c || seq < 0 || seq >= c->lim.max_batch) return -1;
  return c->L[seq];
}

int msd_prefill(msd_ctx* c, int seq, int n, const int32_t* tokens_h, const uint8_t* is_visual_h,
                const void* visual_d, int32_t* first_token_h) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  const msd_model_desc& m = c->m;
  if (seq < 0 || seq >= c->lim.max_batch) return fail(c, MSD_ERR_INVALID_ARG, "bad sequence");
  if (n <= 0 || n > c->lim.max_prompt || !tokens_h || !is_visual_h || !first_token_h)
    return fail(c, MSD_ERR_INVALID_ARG, "bad prompt");
  if (n + c->lim.max_tree > c->lim.max_seq)
    return fail(c, MSD_ERR_CAPACITY, "prompt does not fit the KV cache");
  if (is_visual_h[n - 1]) return fail(c, MSD_ERR_INVALID_ARG, "prompt must end in a text token");
  c->verified_T = 0;  // a prompt invalidates a pending verify (it rewrites the features)
  int n_vis = 0;
  for (int i = 0; i < n; ++i) {
    if (!is_visual_h[i] && (tokens_h[i] < 0 || tokens_h[i] >= m.vocab))
      return fail(c, MSD_ERR_INVALID_ARG, "token id out of range");
    n_vis += is_visual_h[i] ? 1 : 0;
  }
  if (n_vis && !visual_d) return fail(c, MSD_ERR_INVALID_ARG, "visual rows missing");
  TRY(prompt_target(c, seq, n, tokens_h, is_visual_h, visual_d));
  const int d = m.d_model;
  Parts pt;
  TRY(gemm(c, GK_LMHEAD, c->h + (size_t)(n - 1) * 2 * d, 2 * d, 1, c->lm_p, nullptr, m.vocab, d,
           &pt));
  launch_topk(pt, 1, m.vocab, 1, c->tk_idx, c->tk_val, nullptr, nullptr, c->tk_scratch, c->st);
  LAUNCHED(c);
  launch_set_int(c->d_root, seq, c->tk_idx, 0, c->st);
  launch_set_int(c->nxt, n - 1, c->tk_idx, 0, c->st);
  LAUNCHED(c);
  // draft over the prompt: text rows f_down(Concat(h_i, e_{i+1})), visual rows
  // e_i (or h_i for the Visual Feature input)
  launch_fc_input(c->h, nullptr, c->rows.hrow, c->embed, c->nxt, (const uint16_t*)visual_d, n, d,
                  c->fcin, c->st);
  LAUNCHED(c);
  TRY(draft_pass(c, 1, n, -1, n, n_vis ? (const uint16_t*)visual_d : nullptr));
  int st_len[2] = {n, 0};
  TRY(upload_many(c, {{c->d_len + seq, st_len, sizeof(int)}, {c->pend_n + seq, st_len + 1, sizeof(int)}}));
  int* back = c->stage + STAGE_INTS - 64;
  HIPC(c, hipMemcpyAsync(back, c->d_root + seq, sizeof(int), hipMemcpyDeviceToHost, c->st));
  HIPC(c, hipStreamSynchronize(c->st));
  *first_token_h = back[0];
  c->L[seq] = n;
  c->pend[seq] = 0;
  c->ready[seq] = 1;
  return MSD_OK;
}

int msd_set_draft_input(msd_ctx* c, int visual_input) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  if (visual_input != MSD_DRAFT_VISUAL_EMBEDDING && visual_input != MSD_DRAFT_VISUAL_FEATURE)
    return fail(c, MSD_ERR_INVALID_ARG, "unknown draft input mode");
  c->visual_input = visual_input;
  return MSD_OK;
}

int msd_use_caller_weights(msd_ctx* c, int enable) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  c->caller_w = enable != 0;
  return MSD_OK;
}

int msd_set_state(msd_ctx* c, int seq, int L, const void* h_d, int32_t next_token) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  if (seq < 0 || seq >= c->lim.max_batch || !h_d) return fail(c, MSD_ERR_INVALID_ARG, "bad argument");
  if (L < 1 || L + c->lim.max_tree > c->lim.max_seq) return fail(c, MSD_ERR_CAPACITY, "length does not fit");
  if (next_token < 0 || next_token >= c->m.vocab) return fail(c, MSD_ERR_INVALID_ARG, "token out of range");
  c->verified_T = 0;
  int v[4] = {L, next_token, 1, next_token};
  TRY(upload_many(c, {{c->d_len + seq, v, sizeof(int)}, {c->d_root + seq, v + 1, sizeof(int)},
                      {c->pend_n + seq, v + 2, sizeof(int)},
                      {c->pend_next + (size_t)seq * PEND, v + 3, sizeof(int)}}));
  launch_import_row((const uint16_t*)h_d, c->m.d_model,
                    c->pend_h + (size_t)seq * PEND * 2 * c->m.d_model, c->st);
  LAUNCHED(c);
  HIPC(c, hipStreamSynchronize(c->st));
  c->L[seq] = L;
  c->pend[seq] = 1;
  c->ready[seq] = 1;
  return MSD_OK;
}

int msd_draft_tree(msd_ctx* c, int n_seq, const int32_t* seqs_h, const msd_tree_spec* spec,
                   msd_tree* trees_d) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  TRY(check_seqs(c, n_seq, seqs_h));
  if (!spec || !trees_d) return fail(c, MSD_ERR_INVALID_ARG, "null spec or tree buffer");
  c->verified_T = 0;
  const msd_model_desc& m = c->m;
  const int d = m.d_model;
  int T = 0, D = 0, K = 0;
  if (spec->kind == MSD_TREE_STATIC) {
    TRY(prepare_static(c, spec));
    T = c->sp_T;
    D = c->sp_D;
  } else if (spec->kind == MSD_TREE_DYNAMIC) {
    K = spec->topk;
    D = spec->depth;
    T = spec->n_nodes + 1;
    if (K < 1 || K > TOPK || D < 1 || T < 2 || T > c->lim.max_tree || K * (D - 1) > MSD_MAX_TREE ||
        K + (D - 1) * K * K > POOL || spec->n_nodes > K + (D - 1) * K * K)
      return fail(c, MSD_ERR_INVALID_ARG, "bad dynamic tree");
  } else {
    return fail(c, MSD_ERR_INVALID_ARG, "unknown tree kind");
  }
  int max_l = 0, r_max = 0;
  const int region = std::max(T, spec->kind == MSD_TREE_DYNAMIC ? K * (D - 1) : T);
  for (int i = 0; i < n_seq; ++i) {
    const int b = seqs_h[i];
    if (c->L[b] + region > c->lim.max_seq) return fail(c, MSD_ERR_CAPACITY, "KV cache full");
    max_l = std::max(max_l, c->L[b]);
    r_max = std::max(r_max, c->pend[b]);
  }
  TRY(upload_seqs(c, seqs_h, n_seq));
  // 1. catch-up: pending rows through the draft head
  // (a shorter sequence's padding rows write nothing: its region ends at L)
  for (int i = 0; i < n_seq; ++i) {
    c->att_pre[i] = c->L[seqs_h[i]] - c->pend[seqs_h[i]];
    c->att_keys[i] = c->L[seqs_h[i]];
  }
  if (r_max > 0) {
    launch_catchup_next(n_seq, c->seq_ids, c->d_len, c->pend_n, c->pend_next, r_max, PEND, FEAT,
                        c->rows, c->prefix, c->pend_h, c->embed, d, c->fcin, c->st);
    LAUNCHED(c);
    TRY(draft_pass(c, n_seq, r_max, r_max, max_l + r_max, nullptr));
    for (int i = 0; i < n_seq; ++i) c->pend[seqs_h[i]] = 0;
  }
  for (int i = 0; i < n_seq; ++i) c->att_pre[i] = c->L[seqs_h[i]];
  // 2. draft distribution at the root: the last catch-up feature of each
  //    sequence goes through the LM head
  launch_root_feat(n_seq, c->seq_ids, c->dfeat, FEAT, d, c->x, c->xb, c->st);
  LAUNCHED(c);
  if (spec->kind == MSD_TREE_STATIC) {
    TRY(draft_head(c, n_seq, c->round_k[0]));
    launch_tree_init_static(trees_d, n_seq, c->seq_ids, c->d_root, c->sp, T, c->st);
    LAUNCHED(c);
    // round dd expands the depth-dd nodes that have children; its kernel
    // also assigns all depth-dd tokens from the previous round's top-k
    int prev_n = 1, prev_k = c->round_k[0], prev_depth = 0;
    for (int dd = 1; dd < D; ++dd) {
      const int nr = c->round_n[dd];
      if (nr == 0) break;  // no node at this depth has children: none deeper
      launch_static_next(trees_d, n_seq, c->seq_ids, c->d_len, c->sp, T, dd, c->tk_idx, prev_k,
                         prev_n, c->round_off[dd], nr, FEAT, c->rows, c->prefix, c->dfeat,
                         c->embed, d, c->fcin, c->st);
      LAUNCHED(c);
      const int R = c->round_exp_end[dd];
      for (int i = 0; i < n_seq; ++i) c->att_keys[i] = c->L[seqs_h[i]] + R;
      TRY(draft_pass(c, n_seq, nr, R, max_l + R, nullptr));
      TRY(draft_head(c, n_seq * nr, c->round_k[dd]));
      prev_n = nr;
      prev_k = c->round_k[dd];
      prev_depth = dd;
    }
    // the deepest nodes' tokens
    launch_static_assign(trees_d, n_seq, c->sp, T, prev_depth, c->tk_idx, prev_k, prev_n, c->st);
    LAUNCHED(c);
  } else {
    TRY(draft_head(c, n_seq, K));
    launch_dyn_root(c->pool, n_seq, c->tk_idx, c->tk_val, c->tk_lse, K, c->st);
    LAUNCHED(c);
    int n_pool = K, exp_base = K;
    for (int dd = 2; dd <= D; ++dd) {
      launch_dyn_rows(c->pool, n_seq, c->seq_ids, c->d_len, K, dd, FEAT, c->rows, c->prefix, c->st);
      LAUNCHED(c);
      launch_fc_input(nullptr, c->dfeat, c->rows.hrow, c->embed, c->rows.tok, nullptr, n_seq * K,
                      d, c->fcin, c->st);
      LAUNCHED(c);
      const int R = exp_base;
      for (int i = 0; i < n_seq; ++i) c->att_keys[i] = c->L[seqs_h[i]] + R;
      TRY(draft_pass(c, n_seq, K, R, max_l + R, nullptr));
      TRY(draft_head(c, n_seq * K, K));
      launch_dyn_expand(c->pool, n_seq, c->tk_idx, c->tk_val, c->tk_lse, K, n_pool, exp_base, c->st);
      LAUNCHED(c);
      n_pool += K * K;
      exp_base += K;
    }
    launch_dyn_finalize(c->pool, trees_d, n_seq, c->seq_ids, c->d_root, n_pool, T - 1, c->st);
    LAUNCHED(c);
  }
  return MSD_OK;
}

}  // extern "C"

namespace {

// Argument checks of a verify call; *max_l receives the longest committed
// length among the call's sequences.
int check_verify(msd_ctx* c, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d, int T,
                 const int32_t* argmax_d, int* max_l) {
  TRY(check_seqs(c, n_seq, seqs_h));
  if (!trees_d || !argmax_d || T < 1 || T > c->lim.max_tree)
    return fail(c, MSD_ERR_INVALID_ARG, "bad tree");
  *max_l = 0;
  for (int i = 0; i < n_seq; ++i) {
    const int b = seqs_h[i];
    if (c->L[b] + T > c->lim.max_seq) return fail(c, MSD_ERR_CAPACITY, "KV cache full");
    *max_l = std::max(*max_l, c->L[b]);
  }
  return MSD_OK;
}

// The verification itself (checked arguments): the target over every tree's
// nodes, then the LM head with argmax (and the logits when asked).
int verify_impl(msd_ctx* c, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d, int T,
                int max_l, int32_t* argmax_d, float* logits_d) {
  const msd_model_desc& m = c->m;
  const int d = m.d_model, V = m.vocab;
  TRY(upload_seqs(c, seqs_h, n_seq));
  for (int i = 0; i < n_seq; ++i) {
    c->att_pre[i] = c->L[seqs_h[i]];
    c->att_keys[i] = c->L[seqs_h[i]] + T;
  }
  const int rows = n_seq * T;
  c->verified_T = 0;
  launch_verify_rows(trees_d, n_seq, c->seq_ids, c->d_len, T, V, c->rows, c->prefix,
                     c->tree_err, c->st);
  LAUNCHED(c);
  launch_embed(c->embed, c->rows.tok, nullptr, nullptr, rows, d, c->x, c->st);
  LAUNCHED(c);
  TRY(norm_rows(c, rows, c->layers[0].n1));
  TRY(forward_layers(c, false, n_seq, T, T, max_l + T, c->final_norm, c->h, nullptr));
  Parts pt;
  for (int m0 = 0; m0 < rows; m0 += CHUNK) {
    const int mc = std::min(CHUNK, rows - m0);
    TRY(gemm(c, GK_LMHEAD, c->h + (size_t)m0 * 2 * d, 2 * d, mc, c->lm_p, nullptr, V, d, &pt));
    launch_topk(pt, mc, V, 1, argmax_d + m0, nullptr, nullptr,
                logits_d ? logits_d + (size_t)m0 * V : nullptr, c->tk_scratch, c->st);
    LAUNCHED(c);
  }
  c->verified_T = T;
  c->verified_seqs.assign(seqs_h, seqs_h + n_seq);
  return MSD_OK;
}

// Floats of GEMM partials a verify of `rows` tree rows writes (the largest
// of its launches: q/k/v, output, gate+up, down and LM head, for each chunk
// size of CHUNK-row launches).
size_t verify_part_floats(const msd_model_desc& m, int rows) {
  const int d = m.d_model, F = m.ffn_dim, hh = m.n_heads * m.head_dim;
  const int qkv = (m.n_heads + 2 * m.n_kv_heads) * m.head_dim;
  size_t need = 0;
  for (int mc : {std::min(CHUNK, rows), rows % CHUNK}) {
    if (mc <= 0) continue;
    for (size_t f : {gemm_part_floats(mc, qkv, d, 1, GEMM_WGS),
                     gemm_part_floats(mc, d, hh, 1, GEMM_WGS),
                     gemm_part_floats(mc, F, d, 2, GEMM_WGS),
                     gemm_part_floats(mc, d, F, 1, GEMM_WGS),
                     gemm_part_floats(mc, m.vocab, d, 1, GEMM_WGS)})
      need = std::max(need, f);
  }
  return need;
}

}  // namespace

extern "C" {

int msd_verify(msd_ctx* c, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d, int n_nodes,
               int32_t* argmax_d, float* logits_d) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  int max_l = 0;
  TRY(check_verify(c, n_seq, seqs_h, trees_d, n_nodes, argmax_d, &max_l));
  return verify_impl(c, n_seq, seqs_h, trees_d, n_nodes, max_l, argmax_d, logits_d);
}

int msd_verify_noalloc(msd_ctx* c, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d,
                       int n_nodes, int32_t* argmax_d, float* logits_d) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  int max_l = 0;
  TRY(check_verify(c, n_seq, seqs_h, trees_d, n_nodes, argmax_d, &max_l));
  const msd_model_desc& m = c->m;
  const int rows = n_seq * n_nodes;
  if (rows > BIG_MIN_ROWS)
    return fail(c, MSD_ERR_INVALID_ARG,
                "msd_verify_noalloc takes at most " + std::to_string(BIG_MIN_ROWS) +
                    " tree rows per call (n_seq * n_nodes)");
  // the same attention chunking as msd_verify, so both compute identically
  const TreeChunks tc = plan_tree_chunks(m, n_seq, n_nodes, max_l + n_nodes,
                                         c->plan.attn_floats);
  const size_t part = verify_part_floats(m, rows);
  const size_t att_o = tc.part_floats;
  const size_t att_ml = att_o / m.head_dim * 2 + 64;
  const size_t tk = topk_scratch_floats(std::min(CHUNK, rows), m.vocab);
  auto up = [](size_t f) { return (f + 63) / 64 * 64; };  // 256-byte steps
  const size_t need = up(part) + up(att_o) + up(att_ml) + up(tk);
  if (need * sizeof(float) > MSD_NOALLOC_SCRATCH_BYTES)
    return fail(c, MSD_ERR_INVALID_ARG,
                "this verify needs " + std::to_string(need * sizeof(float)) +
                    " bytes of scratch; msd_verify_noalloc holds " +
                    std::to_string((size_t)MSD_NOALLOC_SCRATCH_BYTES));
  // swap the workspace scratch for the static one for this call
  struct Swap {
    msd_ctx* c;
    float *part, *att_po, *att_ml, *tk;
    size_t part_floats, attn_floats;
    ~Swap() {
      c->part = part;
      c->att_po = att_po;
      c->att_ml = att_ml;
      c->tk_scratch = tk;
      c->plan.part_floats = part_floats;
      c->plan.attn_floats = attn_floats;
    }
  } keep{c, c->part, c->att_po, c->att_ml, c->tk_scratch, c->plan.part_floats,
         c->plan.attn_floats};
  float* base = c->noalloc_base;
  c->part = base;
  c->plan.part_floats = part;
  c->att_po = base + up(part);
  c->att_ml = c->att_po + up(att_o);
  c->tk_scratch = c->att_ml + up(att_ml);
  return verify_impl(c, n_seq, seqs_h, trees_d, n_nodes, max_l, argmax_d, logits_d);
}

int msd_accept_compact(msd_ctx* c, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d,
                       int n_nodes, const int32_t* argmax_d, int32_t* emitted_h,
                       int32_t* n_emitted_h, int32_t* slot_map_d) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  TRY(check_accept(c, n_seq, seqs_h, trees_d, n_nodes, emitted_h, n_emitted_h));
  if (!argmax_d) return fail(c, MSD_ERR_INVALID_ARG, "null argument");
  int* slots = slot_map_d ? slot_map_d : c->acc_slot;
  launch_accept(trees_d, n_seq, c->seq_ids, n_nodes, argmax_d, c->acc_path, c->acc_n,
                c->acc_emit, slots, c->d_len, c->tree_err, c->st);
  LAUNCHED(c);
  return finish_accept(c, n_seq, seqs_h, n_nodes, emitted_h, n_emitted_h);
}

int msd_accept_sample(msd_ctx* c, int n_seq, const int32_t* seqs_h, const msd_tree* trees_d,
                      int n_nodes, const float* logits_d, float temperature, uint64_t seed,
                      int32_t* emitted_h, int32_t* n_emitted_h, int32_t* slot_map_d) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  TRY(check_accept(c, n_seq, seqs_h, trees_d, n_nodes, emitted_h, n_emitted_h));
  if (!logits_d) return fail(c, MSD_ERR_INVALID_ARG, "null logits");
  const float inv_t = 1.0f / temperature;
  if (!(temperature > 0.f) || !std::isfinite(temperature) || !std::isfinite(inv_t))
    return fail(c, MSD_ERR_INVALID_ARG, "temperature must be positive and finite");
  for (int i = 0; i < n_seq; ++i)
    if (c->L[seqs_h[i]] >= (1 << 24)) return fail(c, MSD_ERR_INVALID_ARG, "sequence too long");
  int* slots = slot_map_d ? slot_map_d : c->acc_slot;
  launch_accept_sample(trees_d, n_seq, c->seq_ids, n_nodes, logits_d, c->m.vocab, inv_t, seed,
                       c->acc_path, c->acc_n, c->acc_emit, slots, c->d_len, c->tree_err,
                       c->st);
  LAUNCHED(c);
  return finish_accept(c, n_seq, seqs_h, n_nodes, emitted_h, n_emitted_h);
}

int msd_stream_read(const void* buf_d, size_t bytes, int workgroups, void* sink_d,
                    void* stream) {
  const size_t span = stream_span_bytes();
  if (!buf_d || !sink_d || workgroups <= 0 || workgroups > 65536 || bytes < span ||
      bytes % span || ((uintptr_t)buf_d & 15))
    return fail(nullptr, MSD_ERR_INVALID_ARG, "msd_stream_read: bad arguments");
  launch_stream_read(static_cast<const uint16_t*>(buf_d), bytes / span, workgroups,
                     static_cast<unsigned*>(sink_d), (hipStream_t)stream);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(nullptr, MSD_ERR_HIP, hipGetErrorString(e));
  return MSD_OK;
}

int msd_train_accumulate(msd_ctx* c, int seq, int n, const int32_t* tokens_h,
                         const uint8_t* is_visual_h, const void* visual_d, double* loss_h) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  const msd_model_desc& m = c->m;
  if (seq < 0 || seq >= c->lim.max_batch) return fail(c, MSD_ERR_INVALID_ARG, "bad sequence");
  if (n < 2 || n > c->lim.max_prompt || n > c->lim.max_seq || !tokens_h || !is_visual_h ||
      !loss_h)
    return fail(c, MSD_ERR_INVALID_ARG, "bad training sequence");
  int n_vis = 0;
  for (int i = 0; i < n; ++i) {
    if (!is_visual_h[i] && (tokens_h[i] < 0 || tokens_h[i] >= m.vocab))
      return fail(c, MSD_ERR_INVALID_ARG, "token id out of range");
    n_vis += is_visual_h[i] ? 1 : 0;
  }
  if (n_vis && !visual_d) return fail(c, MSD_ERR_INVALID_ARG, "visual rows missing");
  TRY(train_init(c));
  c->verified_T = 0;
  // the slot's cache now holds the training sequence: no longer a decode state
  c->ready[seq] = 0;
  c->L[seq] = 0;
  TRY(prompt_target(c, seq, n, tokens_h, is_visual_h, visual_d));
  return train_pass(c, n, visual_d, loss_h);
}

int msd_train_apply(msd_ctx* c, double lr) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  TrainState* t = c->tr;
  if (!t || t->rows <= 0) return fail(c, MSD_ERR_INVALID_ARG, "no accumulated gradients");
  if (!(lr >= 0.0)) return fail(c, MSD_ERR_INVALID_ARG, "bad learning rate");
  const msd_model_desc& m = c->m;
  const int d = m.d_model, F = m.ffn_dim, H = m.n_heads, KV = m.n_kv_heads, hd = m.head_dim;
  const size_t np = t->off[TRAIN_PARAMS];
  t->steps += 1;
  const float c1 = (float)(1.0 - std::pow((double)ADAM_B1, t->steps));
  const float c2 = (float)(1.0 - std::pow((double)ADAM_B2, t->steps));
  tr_adamw(t->w, t->g, t->m, t->v, np, (float)(1.0 / t->rows), (float)lr, c1, c2, ADAM_B1, ADAM_B2,
           ADAM_EPS, t->wb, c->st);
  LAUNCHED(c);
  // the decoder's packed copies (the norm gains it reads from wb directly)
  const PackedLayer& pl = c->pdlayer;
  const size_t pq = packed_elems(H * hd, d), pk = packed_elems(KV * hd, d);
  uint16_t* qkv = const_cast<uint16_t*>(pl.qkv);
  launch_pack(t->wb + t->off[0], d, 2 * d, const_cast<uint16_t*>(c->fc_p), c->st);
  launch_pack(t->wb + t->off[1], H * hd, d, qkv, c->st);
  launch_pack(t->wb + t->off[2], KV * hd, d, qkv + pq, c->st);
  launch_pack(t->wb + t->off[3], KV * hd, d, qkv + pq + pk, c->st);
  launch_pack(t->wb + t->off[4], d, H * hd, const_cast<uint16_t*>(pl.o), c->st);
  launch_pack(t->wb + t->off[5], F, d, const_cast<uint16_t*>(pl.g), c->st);
  launch_pack(t->wb + t->off[6], F, d, const_cast<uint16_t*>(pl.u), c->st);
  launch_pack(t->wb + t->off[7], d, F, const_cast<uint16_t*>(pl.d), c->st);
  tr_fill(t->g, np, 0.f, c->st);
  LAUNCHED(c);
  t->rows = 0;
  HIPC(c, hipStreamSynchronize(c->st));
  return MSD_OK;
}

int msd_train_read(msd_ctx* c, int what, float* out_d, size_t n_floats) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  TRY(train_init(c));
  TrainState* t = c->tr;
  const size_t np = t->off[TRAIN_PARAMS];
  if (!out_d || n_floats != np)
    return fail(c, MSD_ERR_INVALID_ARG, "msd_train_read wants " + std::to_string(np) + " floats");
  const float* src = what == 0 ? t->g : what == 1 ? t->w : nullptr;
  if (!src) return fail(c, MSD_ERR_INVALID_ARG, "unknown training buffer");
  HIPC(c, hipMemcpyAsync(out_d, src, np * sizeof(float), hipMemcpyDeviceToDevice, c->st));
  HIPC(c, hipStreamSynchronize(c->st));
  return MSD_OK;
}

int msd_train_lr(int step, int total_steps, double lr_max, double* lr_out) {
  if (total_steps <= 0 || step < 0 || step > total_steps || !lr_out)
    return fail(nullptr, MSD_ERR_INVALID_ARG, "bad schedule arguments");
  *lr_out = 0.5 * lr_max * (1.0 + std::cos(M_PI * (double)step / (double)total_steps));
  return MSD_OK;
}

int msd_train_mix(int epoch, int n_epochs, int n_per_epoch, int* n_text_out,
                  int* n_visual_out) {
  if (n_epochs <= 0 || epoch < 0 || epoch > n_epochs || n_per_epoch < 0 || !n_text_out ||
      !n_visual_out)
    return fail(nullptr, MSD_ERR_INVALID_ARG, "bad mix arguments");
  const int nv = (int)std::nearbyint((double)n_per_epoch * epoch / n_epochs);
  *n_visual_out = nv;
  *n_text_out = n_per_epoch - nv;
  return MSD_OK;
}

int msd_trace_enable(msd_ctx* c, int capacity, int kinds) {
  if (!c) return fail(nullptr, MSD_ERR_INVALID_ARG, "null context");
  HIPC(c, hipStreamSynchronize(c->st));
  c->trace.clear();
  if (capacity <= 0) {
    c->tracing = false;
    return MSD_OK;
  }
  while (c->ev_pool.size() < 2 * (size_t)capacity) {
    hipEvent_t e;
    HIPC(c, hipEventCreate(&e));
    c->ev_pool.push_back(e);
  }
  c->trace_cap = (size_t)capacity;
  c->trace_kinds = kinds;
  c->tracing = true;
  return MSD_OK;
}

int msd_trace_read(msd_ctx* c, int max_recs, msd_trace_rec* out) {
  if (!c || (max_recs > 0 && !out)) return fail(c, MSD_ERR_INVALID_ARG, "bad argument");
  HIPC(c, hipStreamSynchronize(c->st));
  const int n = std::min((int)c->trace.size(), max_recs);
  for (int i = 0; i < n; ++i) {
    const msd_ctx::TraceRec& r = c->trace[i];
    float ms = 0.f;
    HIPC(c, hipEventElapsedTime(&ms, r.a, r.b));
    out[i].kind = r.epi;
    out[i].m = r.M;
    out[i].n = r.N;
    out[i].k = r.K;
    out[i].ms = ms;
  }
  return n;
}

}  // extern "C"
