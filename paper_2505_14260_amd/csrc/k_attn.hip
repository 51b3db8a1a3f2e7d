// Attention over the KV cache on gfx950 MFMA.
//
// Tree mode (verification, draft expansion and draft catch-up): every query
// row sees the whole prefix [0, P) of its sequence and the slots of its
// region [P, keys) whose bit is set in its 64-bit mask (tree-structured
// attention of the draft/verify phases; a triangular mask gives causal
// rows); slots at or past keys are never read.  A
// workgroup of 4 waves owns one (sequence, kv head, 32-row query tile, key
// chunk); its waves split the chunk, run an online softmax each, and merge
// their states through LDS into one partial per workgroup; a combine kernel
// merges the chunks in fixed order.  Query rows of a tile are (node,
// head-in-group) pairs so a GQA group shares every K/V load.
// Causal mode (prompt processing): one workgroup per (sequence, head, 32
// consecutive query rows); its waves split the keys up to the diagonal and
// merge through LDS.
//
// Per 32-key block: S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (A = K rows,
// B = Q^T), then O^T += V^T P^T (A = V^T rows of the transposed V cache,
// B = P^T).  The K rows feeding MFMA row i are key pi(i) (bits 2 and 3 of i
// swapped), which makes each lane's eight P values of the second product
// correspond to eight consecutive keys, i.e. one 16-byte load of V^T.
// Q (split rows from the RoPE kernel) and P enter the MFMAs as bf16 hi + lo
// pairs, so only the bf16 cache rows limit the precision; the output rows
// are split rows (the O projection's input).
#include <hip/hip_ext.h>

#include <algorithm>

#include "msd_internal.h"

namespace msd {

namespace {

MSD_DEV int perm_key(int x) { return (x & ~12) | ((x & 4) << 1) | ((x & 8) >> 1); }

MSD_DEV float wave_xor32_max(float v) { return fmaxf(v, __shfl_xor(v, 32)); }
MSD_DEV float wave_xor32_sum(float v) { return v + __shfl_xor(v, 32); }

template <int HD>
struct AttnState {
  f32x16 o[HD / 32];
  float m, l;
};

// K rows of the 32-key block starting at kb for the S^T product (A operand).
// Rows past the cache (S slots) read the last slot instead; their scores
// are replaced by -inf before any use, so whatever those slots hold is never
// seen and the loads need no branch.
template <int HD>
MSD_DEV void load_k(uint4 (&kf)[HD / 16], const uint16_t* kbase, int kb, int S) {
  const int lane = threadIdx.x & 63;
  const int krow = min(kb + perm_key(lane & 31), S - 1);
  const uint16_t* kp = kbase + (size_t)krow * HD + (HD / 2) * (lane >> 5);
#pragma unroll
  for (int c = 0; c < HD / 16; ++c) kf[c] = *reinterpret_cast<const uint4*>(kp + 8 * c);
}

// V^T columns of the block for the O^T product (A operand): eight
// consecutive keys per 16-byte load (S is a multiple of 8).  The clamp keeps
// the address inside the cache; a clamped load only ever covers keys at or
// past S, which mask_v zeroes (S >= k_valid).
template <int HD>
MSD_DEV void load_v(uint4 (&vf)[HD / 32][2], const uint16_t* vbase, int S, int kb) {
  const int lane = threadIdx.x & 63;
  const int i = lane & 31, h = lane >> 5;
#pragma unroll
  for (int dt = 0; dt < HD / 32; ++dt) {
    const uint16_t* vp = vbase + (size_t)(dt * 32 + i) * S;
#pragma unroll
    for (int pk = 0; pk < 2; ++pk)
      vf[dt][pk] = *reinterpret_cast<const uint4*>(vp + min(kb + 16 * pk + 8 * h, S - 8));
  }
}

// The loaded V^T columns with keys at or past k_valid set to zero: their
// probabilities are zero, but the slots may hold any bits (never written, or
// left by the caller), and 0 * NaN would poison the sum.  Applied at the
// point of use so that the loads stay in flight until then.
template <int HD>
MSD_DEV void mask_v(uint4 (&vm)[HD / 32][2], const uint4 (&vf)[HD / 32][2], int kb, int k_valid) {
  const int h = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int pk = 0; pk < 2; ++pk) {
    const int nv = k_valid - (kb + 16 * pk + 8 * h);
    uint32_t keep[4];  // per 32-bit word: keys 2e (low half) and 2e+1 (high half)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      keep[e] = (2 * e + 1 < nv) ? 0xFFFFFFFFu : ((2 * e < nv) ? 0x0000FFFFu : 0u);
#pragma unroll
    for (int dt = 0; dt < HD / 32; ++dt)
      vm[dt][pk] = make_uint4(vf[dt][pk].x & keep[0], vf[dt][pk].y & keep[1],
                              vf[dt][pk].z & keep[2], vf[dt][pk].w & keep[3]);
  }
}

// Two floats as packed bfloat16, rounded to nearest even (one
// v_cvt_pk_bf16_f32 on gfx950).
MSD_DEV uint32_t pack_bf16(float a, float b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)b) << 16);
}

// The running maximum that scales a column's exponentials is raised only
// when a block's maximum exceeds it by more than this (natural-log units),
// so most blocks skip rescaling the output; the exponentials then stay below
// e^8, far inside float and bfloat16 range.  Any reference gives the same
// normalised result.
constexpr float RESCALE_SLACK = 8.f;

// Online-softmax accumulation of keys [k_begin, k_end) (k_begin a multiple
// of 32) for the 32 query columns of the wave; qf(c, lo) returns the lane's
// bf16 hi (lo = 0) or lo (lo = 1) query fragment of MFMA step c, and
// vis(key) says whether the lane's query sees the key.  Keys at or past
// k_valid (>= k_end) are never taken from the cache.  Each block's K rows are
// reloaded with the next block as soon as the score MFMAs have consumed them,
// the V columns as soon as the output MFMAs have; the last block reloads
// itself (a cache hit) so the loop has no branch around its loads.  kf and
// vf arrive holding the block at k_begin (attend_prefetch), so the caller can
// issue those loads before its own set-up.
template <int HD>
MSD_DEV void attend_prefetch(uint4 (&kf)[HD / 16], uint4 (&vf)[HD / 32][2],
                             const uint16_t* kbase, const uint16_t* vbase, int S, int k_begin) {
  load_k<HD>(kf, kbase, k_begin, S);
  load_v<HD>(vf, vbase, S, k_begin);
}

template <int HD, typename QF, typename Vis>
MSD_DEV void attend_range(AttnState<HD>& st, QF qf, uint4 (&kf)[HD / 16],
                          uint4 (&vf)[HD / 32][2], const uint16_t* kbase,
                          const uint16_t* vbase, int S, int k_begin, int k_end, int k_valid,
                          float scale, Vis vis) {
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5;
  if (k_begin >= k_end) return;
  const int k_last = k_begin + ((k_end - 1 - k_begin) & ~31);
  bool fresh = true;  // the output state is still all zero
  for (int kb = k_begin; kb < k_end; kb += 32) {
    const int nb = min(kb + 32, k_last);
    // ---- S^T tile: rows = keys, columns = query rows
    f32x16 s = {};
#pragma unroll
    for (int c = 0; c < HD / 16; ++c) {
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[c]), qf(c, 0), s, 0, 0, 0);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[c]), qf(c, 1), s, 0, 0, 0);
    }
    load_k<HD>(kf, kbase, nb, S);
    float bm = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = kb + perm_key(8 * (r >> 2) + 4 * h + (r & 3));
      const bool ok = (key < k_end) & vis(key);
      s[r] = ok ? s[r] * scale : -INFINITY;
      bm = fmaxf(bm, s[r]);
    }
    bm = wave_xor32_max(bm);
    const bool raise = bm > st.m + RESCALE_SLACK;  // also when st.m is still -inf
    if (__any(raise)) {
      const float m_new = raise ? bm : st.m;
      if (!fresh) {
        const float alpha = (st.m == -INFINITY) ? 0.f : __expf(st.m - m_new);
        st.l *= alpha;
#pragma unroll
        for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) st.o[dt][r] *= alpha;
      }
      st.m = m_new;
    }
    fresh = false;
    float p[16];
    float rs = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = (st.m == -INFINITY) ? 0.f : __expf(s[r] - st.m);
      rs += p[r];
    }
    st.l += wave_xor32_sum(rs);
    // P as bf16 hi + lo pairs
    uint4 pb[2], pl[2];
#pragma unroll
    for (int pk = 0; pk < 2; ++pk) {
      uint32_t w[4], wl[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = p[pk * 8 + 2 * e], p1 = p[pk * 8 + 2 * e + 1];
        w[e] = pack_bf16(p0, p1);
        wl[e] = pack_bf16(p0 - __uint_as_float(w[e] << 16), p1 - __uint_as_float(w[e] & 0xFFFF0000u));
      }
      pb[pk] = make_uint4(w[0], w[1], w[2], w[3]);
      pl[pk] = make_uint4(wl[0], wl[1], wl[2], wl[3]);
    }
    // ---- O^T += V^T P^T
    uint4 vm[HD / 32][2];
    mask_v<HD>(vm, vf, kb, k_valid);
    load_v<HD>(vf, vbase, S, nb);
#pragma unroll
    for (int dt = 0; dt < HD / 32; ++dt) {
#pragma unroll
      for (int pk = 0; pk < 2; ++pk) {
        st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vm[dt][pk]), as_bf16x8(pb[pk]),
                                                           st.o[dt], 0, 0, 0);
        st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vm[dt][pk]), as_bf16x8(pl[pk]),
                                                           st.o[dt], 0, 0, 0);
      }
    }
  }
}

// The lane's 8-element slices of its query row (hi at q[k], lo at q[lo + k]).
template <int HD>
MSD_DEV void load_q(bf16x8 (&qh)[HD / 16], bf16x8 (&ql)[HD / 16], const uint16_t* qrow, int lo) {
  const int h = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int c = 0; c < HD / 16; ++c) {
    qh[c] = as_bf16x8(*reinterpret_cast<const uint4*>(qrow + (HD / 2) * h + 8 * c));
    ql[c] = as_bf16x8(*reinterpret_cast<const uint4*>(qrow + lo + (HD / 2) * h + 8 * c));
  }
}

template <int HD>
MSD_DEV void init_state(AttnState<HD>& st) {
#pragma unroll
  for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) st.o[dt][r] = 0.f;
  st.m = -INFINITY;
  st.l = 0.f;
}

// O^T C layout: lane holds query column (lane & 31), register r of dim tile
// dt holds dim dt*32 + 8*(r/4) + 4*(lane/32) + r%4.
template <int HD>
MSD_DEV void store_final(const AttnState<HD>& st, uint16_t* orow, int K, bool valid) {
  if (!valid) return;
  const int h = (threadIdx.x & 63) >> 5;
  const float inv = st.l > 0.f ? 1.f / st.l : 0.f;
#pragma unroll
  for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      put_split(orow, K, dt * 32 + 8 * (r >> 2) + 4 * h + (r & 3), st.o[dt][r] * inv);
}

// Output element e of a wave's state: register e / 64 of lane e % 64, i.e.
// query column (e % 64) & 31 and head dim dim_of(e).
template <int HD>
MSD_DEV int dim_of(int e) {
  const int R = e >> 6, L = e & 63;
  const int dt = R >> 4, r = R & 15;
  return dt * 32 + 8 * (r >> 2) + 4 * (L >> 5) + (r & 3);
}

// Inverse of dim_of: the state element of query column j and head dim d.
template <int HD>
MSD_DEV int state_index(int j, int d) {
  const int dt = d >> 5, w = d & 31;
  const int r = 4 * (w >> 3) + (w & 3), hh = (w >> 2) & 1;
  return (dt * 16 + r) * 64 + j + 32 * hh;
}

// Eight consecutive values of a split row: hi halves at row[0..8), lo halves
// at row[lo..lo+8), one 16-byte store each (row 16-byte aligned).
MSD_DEV void store_split8(uint16_t* row, int lo, const float (&v)[8]) {
  uint32_t hw[4], lw[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    hw[e] = pack_bf16(v[2 * e], v[2 * e + 1]);
    lw[e] = pack_bf16(v[2 * e] - __uint_as_float(hw[e] << 16),
                      v[2 * e + 1] - __uint_as_float(hw[e] & 0xFFFF0000u));
  }
  *reinterpret_cast<uint4*>(row) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
  *reinterpret_cast<uint4*>(row + lo) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
}

// Query column j of tile qt -> (node, head); node >= nq marks padding.
MSD_DEV void column_to_row(int qt, int j, int G, int g, int& node, int& head) {
  const int qr = qt * 32 + j;
  node = qr / G;
  head = g * G + (qr - node * G);
}

// Query fragments of the causal kernel, held in registers.
template <int HD>
struct QRegs {
  const bf16x8* h;
  const bf16x8* l;
  MSD_DEV bf16x8 operator()(int c, int lo) const { return lo ? l[c] : h[c]; }
};

// Query fragments of the tree kernel, read from the workgroup's LDS copy:
// column j holds its hi then lo halves in 16-byte units, unit u at
// j * QU + (u ^ (j & 15)) so that 16 lanes reading the same unit of 16
// different columns hit different banks.
template <int HD>
struct QShared {
  static constexpr int QU = HD / 4;  // 16-byte units per column
  const uint4* col;                  // the lane's column
  int sw;                            // j & 15
  int h;                             // lane / 32
  MSD_DEV bf16x8 operator()(int c, int lo) const {
    const int u = lo * (HD / 8) + (HD / 16) * h + c;
    return as_bf16x8(col[u ^ sw]);
  }
};

// A chunk's partial output is stored normalised by its own softmax sum (a
// convex combination of value rows, so no larger in magnitude than the
// largest of them) in float16, eight head dims per 16-byte unit; its
// (max, sum) pair stays float32.
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
MSD_DEV uint4 pack_half8(const float (&o)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = __builtin_bit_cast(uint32_t, half2v{(_Float16)o[2 * i], (_Float16)o[2 * i + 1]});
  return make_uint4(w[0], w[1], w[2], w[3]);
}
MSD_DEV float half_lo(uint32_t w) { return (float)__builtin_bit_cast(half2v, w).x; }
MSD_DEV float half_hi(uint32_t w) { return (float)__builtin_bit_cast(half2v, w).y; }

// Merges the key chunks of one item (sequence, kv head, query tile): run by
// the workgroup that finishes the item's last chunk.  A chunk's partial is
// stored by units of (query column j, 8 consecutive head dims d0..d0+7) at
// ((d0 / 8) * 32 + j) * 8; a thread owns such units: it loads every chunk's
// slices first, then the (max, sum) pairs, so the merge waits for memory
// once, and writes each unit as one 16-byte hi and one 16-byte lo store.
// Chunk q's weight is exp(max_q - max) * sum_q over the total; chunks merge
// in chunk order, so the result does not depend on which workgroup merges.
template <int HD, int NWV>
MSD_DEV void combine_chunks(const AttnArgs& a, size_t item0, int nc, int qt, int g, int sidx,
                            float (*wgt)[32], float* inv_den) {
  constexpr int E = 32 * HD;
  constexpr int NT = 64 * NWV;
  constexpr int UN = 32 * HD / 8;           // (column, 8 dims) units
  constexpr int IT = (UN + NT - 1) / NT;    // units per thread
  const int G = a.H / a.KV;
  uint4 v[IT][ATT_MAX_CHUNKS];
  const uint16_t* const po = reinterpret_cast<const uint16_t*>(a.part_o);
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int u = min((int)threadIdx.x + NT * it, UN - 1);
#pragma unroll
    for (int q = 0; q < ATT_MAX_CHUNKS; ++q)
      v[it][q] = *reinterpret_cast<const uint4*>(po + (item0 + min(q, nc - 1)) * E + 8 * u);
  }
  if (threadIdx.x < 32) {
    const int j = threadIdx.x;
    float2 ml[ATT_MAX_CHUNKS];
#pragma unroll
    for (int q = 0; q < ATT_MAX_CHUNKS; ++q)
      ml[q] = *reinterpret_cast<const float2*>(a.part_ml + (item0 + min(q, nc - 1)) * 64 + 2 * j);
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < ATT_MAX_CHUNKS; ++q)
      if (q < nc) M = fmaxf(M, ml[q].x);
    float den = 0.f;
#pragma unroll
    for (int q = 0; q < ATT_MAX_CHUNKS; ++q) {
      const float wc = (q >= nc || M == -INFINITY || ml[q].x == -INFINITY) ? 0.f
                                                                            : __expf(ml[q].x - M);
      wgt[q][j] = wc * ml[q].y;
      den += wc * ml[q].y;
    }
    inv_den[j] = den > 0.f ? 1.f / den : 0.f;
  }
  lds_barrier();
  const int HH = a.H * HD;
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int u = threadIdx.x + NT * it;
    if (u >= UN) break;
    const int j = u & 31, d0 = 8 * (u >> 5);
    int nd, hd_;
    column_to_row(qt, j, G, g, nd, hd_);
    if (nd >= a.nq) continue;
    float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < ATT_MAX_CHUNKS; ++q) {
      const float wq = wgt[q][j];
      const uint4 h = v[it][q];
      o[0] += wq * half_lo(h.x);
      o[1] += wq * half_hi(h.x);
      o[2] += wq * half_lo(h.y);
      o[3] += wq * half_hi(h.y);
      o[4] += wq * half_lo(h.z);
      o[5] += wq * half_hi(h.z);
      o[6] += wq * half_lo(h.w);
      o[7] += wq * half_hi(h.w);
    }
    const float inv = inv_den[j];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] *= inv;
    store_split8(a.out + (size_t)(sidx * a.nq + nd) * 2 * HH + (size_t)hd_ * HD + d0, HH, o);
  }
}

// Two waves per SIMD (two 4-wave workgroups per CU): the registers stay
// within 256 per lane.
template <int HD, int NWV>
__global__ __launch_bounds__(64 * NWV, 2) void k_tree_attn(AttnArgs a) {
  constexpr int E = 32 * HD;                 // state elements of one wave
  constexpr int QU = QShared<HD>::QU;
  constexpr int NT = 64 * NWV;
  // the query tile lives in the merge buffer's space until the key loop ends
  __shared__ float so[NWV * E];
  static_assert(32 * QU * 4 <= NWV * E, "query tile must fit the merge buffer");
  uint4* const sq = reinterpret_cast<uint4*>(so);
  __shared__ float sml[NWV][32][2];
  __shared__ float wgt[ATT_MAX_CHUNKS > NWV ? ATT_MAX_CHUNKS : NWV][32];
  __shared__ float colm[32][2];
  __shared__ int last;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // Workgroup -> (sequence, kv head) pair, key chunk c and query tile qt.
  // Every workgroup of one item (pair, qt) runs on one XCD (workgroup i runs
  // on XCD i mod 8): its chunks meet in that XCD's L2 for the merge.  With
  // fewer pairs than XCDs a pair's query tiles are dealt over a.xrep XCDs
  // (virtual pair pair * xrep + qt mod xrep), so that every XCD works; the
  // tiles on one XCD (consecutive slots) read the same K/V blocks, fetched
  // from HBM once per XCD.  Grid: 8 * ceil(pairs * xrep / 8) * chunks *
  // ceil(qtiles / xrep).
  const int D = a.xrep;
  const int QD = (a.qtiles + D - 1) / D;  // query tiles per virtual pair
  const int per_pair = QD * a.n_chunks;
  const int slot = blockIdx.x >> 3;
  const int pp = slot / per_pair, rem = slot - pp * per_pair;
  const int vpair = pp * 8 + (blockIdx.x & 7);
  if (vpair >= a.n_seq * a.KV * D) return;
  const int pair = vpair / D;
  const int c = rem / QD, qt = (rem - c * QD) * D + vpair % D;
  if (qt >= a.qtiles) return;
  const int g = pair % a.KV;
  const int sidx = pair / a.KV;
  const int b = a.seq[sidx];
  const int P = a.prefix[sidx];
  const int Ltot = a.keys[sidx];
  const int G = a.H / a.KV;
  const int HH = a.H * HD;
  const uint16_t* kbase = a.kc + (size_t)(b * a.KV + g) * a.S * HD;
  const uint16_t* vbase = a.vc + (size_t)(b * a.KV + g) * HD * a.S;
  const int wk = a.chunk_keys / NWV;
  const int k0 = c * a.chunk_keys + w * wk;
  const int k1 = min(k0 + wk, Ltot);
  // the tile's 32 query columns (hi and lo halves) into LDS; padding
  // columns copy node 0 (their results are dropped).  The query loads go out
  // first, then the first key block's, so that the query staging waits for
  // the query loads only.
  constexpr int QN = 32 * QU / NT;  // 16-byte units per thread
  static_assert(QN * NT == 32 * QU, "query units must divide over the threads");
  uint4 qv[QN];
  int qi[QN];
#pragma unroll
  for (int r = 0; r < QN; ++r) {
    const int u = threadIdx.x + r * NT;
    const int j = u / QU, v = u - j * QU;
    int node, head;
    column_to_row(qt, j, G, g, node, head);
    if (node >= a.nq) { node = 0; head = g * G; }
    const int half = v / (HD / 8), k8 = v - half * (HD / 8);
    qi[r] = j * QU + (v ^ (j & 15));
    qv[r] = *reinterpret_cast<const uint4*>(
        a.q + (size_t)(sidx * a.nq + node) * 2 * HH + (size_t)half * HH + (size_t)head * HD + 8 * k8);
  }
  uint4 kf[HD / 16], vf[HD / 32][2];
  attend_prefetch<HD>(kf, vf, kbase, vbase, a.S, k0);
#pragma unroll
  for (int r = 0; r < QN; ++r) sq[qi[r]] = qv[r];
  int node, head;
  column_to_row(qt, lane & 31, G, g, node, head);
  if (node >= a.nq) node = 0;
  const uint64_t msk = a.mask[sidx * a.nq + node];
  AttnState<HD> st;
  init_state<HD>(st);
  lds_barrier();
  const QShared<HD> qf{sq + (lane & 31) * QU, lane & 15, lane >> 5};
  attend_range<HD>(st, qf, kf, vf, kbase, vbase, a.S, k0, k1, Ltot, a.scale, [&](int key) {
    return (key < P) | (((msk >> ((key - P) & 63)) & 1ull) != 0);
  });
  lds_barrier();  // every wave is done with the query tile
  // merge the waves' states
#pragma unroll
  for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) so[w * E + (dt * 16 + r) * 64 + lane] = st.o[dt][r];
  if (lane < 32) {
    sml[w][lane][0] = st.m;
    sml[w][lane][1] = st.l;
  }
  lds_barrier();
  // per-column merge weights: wgt[q][j] = exp(m_q - M_j)
  if (threadIdx.x < 32) {
    const int j = threadIdx.x;
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < NWV; ++q) M = fmaxf(M, sml[q][j][0]);
    float l = 0.f;
#pragma unroll
    for (int q = 0; q < NWV; ++q) {
      const float mq = sml[q][j][0];
      const float wq = (M == -INFINITY || mq == -INFINITY) ? 0.f : __expf(mq - M);
      wgt[q][j] = wq;
      l += wq * sml[q][j][1];
    }
    colm[j][0] = M;
    colm[j][1] = l;
  }
  lds_barrier();
  if (a.n_chunks == 1) {
    // thread -> (query column j, 8 consecutive dims): one 16-byte store each
    // for the hi and lo halves of the output row
    for (int u = threadIdx.x; u < 32 * (HD / 8); u += NT) {
      const int j = u & 31, d0 = 8 * (u >> 5);
      int nd, hd_;
      column_to_row(qt, j, G, g, nd, hd_);
      if (nd >= a.nq) continue;
      const float l = colm[j][1];
      const float inv = l > 0.f ? 1.f / l : 0.f;
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int e = state_index<HD>(j, d0 + i);
        float o = 0.f;
#pragma unroll
        for (int q = 0; q < NWV; ++q) o += wgt[q][j] * so[q * E + e];
        v[i] = o * inv;
      }
      store_split8(a.out + (size_t)(sidx * a.nq + nd) * 2 * HH + (size_t)hd_ * HD + d0, HH, v);
    }
    return;
  }
  const size_t item = ((size_t)sidx * a.KV + g) * a.qtiles + qt;
  const size_t item0 = item * a.n_chunks;
  // the chunk's partial by units (column j, dims d0..d0+7) at 8 u with
  // u = (d0 / 8) * 32 + j: consecutive threads take consecutive columns
  // (distinct LDS banks) and write consecutive 32-byte units
  for (int u = threadIdx.x; u < 32 * (HD / 8); u += NT) {
    const int j = u & 31, d0 = 8 * (u >> 5);
    const float l = colm[j][1];
    const float inv = l > 0.f ? 1.f / l : 0.f;
    float o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int e = state_index<HD>(j, d0 + i);
      float x = 0.f;
#pragma unroll
      for (int q = 0; q < NWV; ++q) x += wgt[q][j] * so[q * E + e];
      o[i] = x * inv;
    }
    uint16_t* dst = reinterpret_cast<uint16_t*>(a.part_o) + (item0 + c) * E + 8 * u;
    *reinterpret_cast<uint4*>(dst) = pack_half8(o);
  }
  if (threadIdx.x < 32) {
    a.part_ml[(item0 + c) * 64 + 2 * threadIdx.x] = colm[threadIdx.x][0];
    a.part_ml[(item0 + c) * 64 + 2 * threadIdx.x + 1] = colm[threadIdx.x][1];
  }
  // The workgroup that finishes the item's last chunk merges them.  Every
  // chunk of the item runs on this XCD, so its partial is in this XCD's L2
  // once the stores are acknowledged: each thread waits for its own, the
  // barrier for all, and the arrival count is taken after that.  The count
  // keeps one 4-bit field per XCD (read from the XCC_ID hardware register),
  // so the last arrival also sees whether every chunk ran on one XCD; if
  // not, the merge may have read another L2's stale lines and place_err is
  // raised for the host to report.
  __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();
  if (threadIdx.x == 0) {
    unsigned xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const unsigned mine = 1u << (4 * (xcc & 7));
    const unsigned now = __hip_atomic_fetch_add(reinterpret_cast<unsigned*>(a.att_cnt + item), mine,
                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) +
                         mine;
    int total = 0, xcds = 0;
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      const int n = (now >> (4 * x)) & 15;
      total += n;
      xcds += n != 0;
    }
    last = total == a.n_chunks;
    if (last && xcds != 1) __hip_atomic_store(a.place_err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  lds_barrier();
  if (!last) return;
  combine_chunks<HD, NWV>(a, item0, a.n_chunks, qt, g, sidx, wgt, &colm[0][0]);
  if (threadIdx.x == 0)
    __hip_atomic_store(a.att_cnt + item, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Causal attention of a prompt: one workgroup of CAUSAL_WAVES waves per
// (sequence, head, 32-row query tile).  The tile's key blocks [0, end of its
// last row) are split into contiguous quarters, one per wave, each with its
// own online softmax; the waves' states merge through LDS (weights
// exp(m_w - max)) and the workgroup writes the tile's output rows.  Tiles
// are dealt longest first (the last query tiles see the most keys).
constexpr int CAUSAL_WAVES = 4;
template <int HD>
__global__ __launch_bounds__(64 * CAUSAL_WAVES, 2) void k_causal_attn(AttnArgs a) {
  constexpr int NWV = CAUSAL_WAVES;
  constexpr int E = 32 * HD;  // state elements of one wave
  __shared__ float so[NWV * E];
  __shared__ float sml[NWV][32][2];
  __shared__ float wgt[NWV][32];
  __shared__ float colm[32];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n_sh = a.n_seq * a.H;
  const int qt = a.qtiles - 1 - (int)blockIdx.x / n_sh;  // longest tiles first
  const int sh = (int)blockIdx.x % n_sh;
  const int head = sh % a.H;
  const int sidx = sh / a.H;
  const int b = a.seq[sidx];
  const int P = a.prefix[sidx];
  const int g = head / (a.H / a.KV);
  const int j = lane & 31;
  int node = qt * 32 + j;
  const bool valid = node < a.nq;
  if (!valid) node = a.nq - 1;
  const int HH = a.H * HD;
  bf16x8 qh[HD / 16], ql[HD / 16];
  load_q<HD>(qh, ql, a.q + (size_t)(sidx * a.nq + node) * 2 * HH + (size_t)head * HD, HH);
  const uint16_t* kbase = a.kc + (size_t)(b * a.KV + g) * a.S * HD;
  const uint16_t* vbase = a.vc + (size_t)(b * a.KV + g) * HD * a.S;
  const int last = min(qt * 32 + 32, a.nq);
  const int k1 = P + last;  // keys of the tile: [0, k1)
  const int nb = (k1 + 31) / 32;
  const int per = (nb + NWV - 1) / NWV;
  const int kb0 = min(w * per, nb) * 32;
  const int kb1 = min(kb0 + per * 32, k1);
  const int my_last = P + node;
  AttnState<HD> st;
  init_state<HD>(st);
  uint4 kf[HD / 16], vf[HD / 32][2];
  attend_prefetch<HD>(kf, vf, kbase, vbase, a.S, min(kb0, ((k1 - 1) / 32) * 32));
  attend_range<HD>(st, QRegs<HD>{qh, ql}, kf, vf, kbase, vbase, a.S, kb0, kb1, k1, a.scale,
                   [&](int key) { return key <= my_last; });
  // merge the waves' states
#pragma unroll
  for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) so[w * E + (dt * 16 + r) * 64 + lane] = st.o[dt][r];
  if (lane < 32) {
    sml[w][lane][0] = st.m;
    sml[w][lane][1] = st.l;
  }
  lds_barrier();
  if (threadIdx.x < 32) {
    const int jj = threadIdx.x;
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < NWV; ++q) M = fmaxf(M, sml[q][jj][0]);
    float l = 0.f;
#pragma unroll
    for (int q = 0; q < NWV; ++q) {
      const float mq = sml[q][jj][0];
      const float wq = (M == -INFINITY || mq == -INFINITY) ? 0.f : __expf(mq - M);
      wgt[q][jj] = wq;
      l += wq * sml[q][jj][1];
    }
    colm[jj] = l > 0.f ? 1.f / l : 0.f;
  }
  lds_barrier();
  // thread -> (query column jj, 8 consecutive dims): one 16-byte store each
  // for the hi and lo halves of the output row
  for (int u = threadIdx.x; u < 32 * (HD / 8); u += 64 * NWV) {
    const int jj = u & 31, d0 = 8 * (u >> 5);
    const int nd = qt * 32 + jj;
    if (nd >= a.nq) continue;
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int e = state_index<HD>(jj, d0 + i);
      float o = 0.f;
#pragma unroll
      for (int q = 0; q < NWV; ++q) o += wgt[q][jj] * so[q * E + e];
      v[i] = o * colm[jj];
    }
    store_split8(a.out + (size_t)(sidx * a.nq + nd) * 2 * HH + (size_t)head * HD + d0, HH, v);
  }
}

}  // namespace

size_t attn_partial_floats(int n_seq, int KV, int qtiles, int n_chunks, int hd) {
  return (size_t)n_seq * KV * qtiles * n_chunks * 32 * hd;
}

template <int HD>
void launch_tree_hd(AttnArgs a, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  const int pairs = a.n_seq * a.KV;
  // XCDs per pair: the query tiles of fewer than eight pairs are dealt over
  // the idle XCDs (their K/V is then read from HBM once per XCD)
  a.xrep = std::max(1, std::min(8 / pairs, a.qtiles));
  const int QD = (a.qtiles + a.xrep - 1) / a.xrep;
  const dim3 grid(8 * ((pairs * a.xrep + 7) / 8) * QD * a.n_chunks);
  if (ev0)  // events carried by the launch itself bracket the kernel only
    hipExtLaunchKernelGGL((k_tree_attn<HD, TREE_WAVES>), grid, dim3(64 * TREE_WAVES), 0, st,
                          ev0, ev1, 0, a);
  else
    hipLaunchKernelGGL((k_tree_attn<HD, TREE_WAVES>), grid, dim3(64 * TREE_WAVES), 0, st, a);
}

void launch_tree_attention(AttnArgs a, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  if (a.hd == 128) launch_tree_hd<128>(a, st, ev0, ev1);
  else launch_tree_hd<64>(a, st, ev0, ev1);
}

void launch_causal_attention(AttnArgs a, hipStream_t st) {
  const int items = a.n_seq * a.H * a.qtiles;
  dim3 grid(items);
  if (a.hd == 128)
    hipLaunchKernelGGL(k_causal_attn<128>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_causal_attn<64>, grid, dim3(256), 0, st, a);
}

}  // namespace msd
