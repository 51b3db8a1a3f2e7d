// Thin-M GEMM on gfx950 MFMA: P_s[m][n] = sum_{k in chunk s} X[m][k] * W[n][k],
// W in bfloat16 (packed, see below), X as split rows (bf16 hi + lo).
//
// The decode path multiplies a few dozen activation rows (tree nodes) by
// large weight matrices, so the kernel is bound by streaming W from HBM once.
//
// Packed weights.  A weight [N][K] is stored as 64-row tiles times 128-column
// blocks, each block 16 KB in the exact order the four waves of a workgroup
// consume it: block (t, kb) at element ((t * nkt) + kb) * 8192, inside it
// ((wave * 4 + c) * 64 + lane) * 8 + e holds W[t*64 + wave*16 + (lane & 15)]
// [kb*128 + 32*(lane >> 4) + 8*c + e].  Rows past N and columns past K are
// zero.  Every wave load is then 1 KB contiguous and every workgroup streams
// 64 KB spans, read with non-temporal buffer loads (WStream below).  Within
// one MFMA the K index may
// be any permutation shared by the two operands; the X fragments use the same
// permutation.
//
// Work split.  K is cut into chunks of NKB blocks; a workgroup (4 waves) owns
// one chunk and a strided set of tiles, stages its X chunk in LDS once
// (XOR-swizzled, hi halves then lo halves) and then streams the W blocks of
// its tiles through a ring of P register stages: having consumed a block it
// loads the block P places further in its (tile, block) sequence.  The loop
// has no branch on the data path and stores each tile's partial
// unconditionally (padded rows go to a small sink), which keeps every weight
// load in flight across tile boundaries.  Partials part[s][m][n] (float32) are summed in chunk order by
// the kernel that consumes the product, so the result is deterministic.
//
// X arrives split by its producer, x = hi + lo with hi = bf16(x) and
// lo = bf16(x - hi), so W x = W hi + W lo carries about 16 significant bits of
// the activations (one bf16 rounding of every GEMM input, amplified by a deep
// stack of layers, is far larger than the error of the weights' products).
#include <hip/hip_ext.h>

#include "msd_internal.h"

namespace msd {

namespace {

constexpr int KB = 128;       // K elements per block
constexpr int TILE_ROWS = 64;  // 4 waves x 16 rows
constexpr int BLOCK_ELEMS = TILE_ROWS * KB;
// 128-column blocks per K chunk: 8 for up to 32 rows (X chunk 64 or 128 KB
// of LDS), 4 for 64 rows.  Longer chunks mean fewer partials to write and
// re-read; the ring depth stays at RING blocks either way.
constexpr int RING = 4;
__host__ __device__ constexpr int chunk_blocks(int MT) { return MT <= 2 ? 8 : 4; }
constexpr int PAIR_MAX_TILES = 5;  // tiles per workgroup of the two-chunk kernel
// tiles per workgroup of the full-K kernel (k_gemm_fk): launched with 8 or
// 10 (the registers of twelve tiles' accumulators spill)
constexpr int FK_MIN_TILES = 8, FK_MAX_TILES = 10;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
MSD_DEV uint4 load_stream(const uint16_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// The weight stream of the thin GEMMs: raw buffer loads (32-bit data
// format, stride 0) over one packed weight of `bytes` bytes, with the
// non-temporal cache policy.  An element offset e < 0 reads 16 zero bytes:
// the offset 2^31 lies past the buffer's range, so the load is answered
// without a memory access (the ring's slots after the last tile and past K).
// Measured at the 7B verify against the same stream as global loads: plain
// or device/system-scope policies (sc1, sc0 sc1) 3.90 ms, non-temporal
// global loads 3.71 ms, these 3.69 ms (draft 0.888 -> 0.877 ms).
constexpr int WLOAD_POLICY = 2;  // nt; bit 0 would be sc0, bit 4 sc1
struct WStream {
  __amdgpu_buffer_rsrc_t r;
  MSD_DEV WStream(const uint16_t* base, int bytes)
      : r(__builtin_amdgcn_make_buffer_rsrc((void*)base, 0, bytes, 0x00020000)) {}
  // e: element offset (a packed weight holds fewer than 2^30 elements)
  MSD_DEV uint4 load(int e) const {
    const int off = e >= 0 ? e * 2 : (int)0x80000000u;
    const u32x4 v = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, WLOAD_POLICY));
    return make_uint4(v.x, v.y, v.z, v.w);
  }
};

// LDS X chunk: row m holds the chunk's columns in 16-byte units (8 bf16);
// unit u of row m is stored at u ^ (m & 15) so that the 16 rows read by one
// MFMA operand load hit different banks.
MSD_DEV int xs_index(int m, int u, int upr) { return m * upr + (u ^ (m & 15)); }

// MS (row split): a pass of 33-64 rows runs as two 32-row halves.  Workgroups
// b and b + 8 (same XCD) take the two halves of one (chunk, tile set), so
// the second one's weight blocks are L2 hits, and each workgroup streams its
// weight blocks against a 32-row X chunk twice as long as a 64-row one.
template <int MT, int NW, int NKB, int P, bool MS = false>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  static_assert(NKB % P == 0, "ring slots must divide the chunk");
  extern __shared__ uint4 xs[];
  constexpr int UPR = NKB * KB / 8;  // 16-byte units per LDS row
  constexpr int LO = MT * 16 * UPR;  // offset of the lo halves
  constexpr int NX = MT * 16 * UPR / 256;
  constexpr int XB = NX < 16 ? NX : 16;  // staging batch (loads in flight)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, g = lane >> 4;
  const int S = a.S, G = a.G, K = a.K, nkt = a.nkt, n_tiles = a.n_tiles;
  int unit = blockIdx.x, half = 0;
  if (MS) {
    half = (unit >> 3) & 1;
    unit = ((unit >> 4) << 3) | (unit & 7);
    if (unit >= S * G) return;
  }
  const int M = MS ? min(MT * 16, a.M - MT * 16 * half) : a.M;
  const int s = unit % S, gi = unit / S;
  const int n_my = gi < n_tiles ? (n_tiles - gi + G - 1) / G : 0;
  if (n_my == 0) return;
  const int kb0 = s * NKB;
  const int k0 = kb0 * KB;
  const uint16_t* const W = a.W;
  const uint16_t* const W2 = a.W2;
  const int lane_off = wave * (BLOCK_ELEMS / 4) + lane * 8;
  const int tstride = nkt * BLOCK_ELEMS;
  // the chunk's blocks; past K (last chunk) the loads read zeros, X being
  // zero there too
  const int nvb = min(NKB, nkt - kb0);

  // X[0:MT*16, k0:k0+NKB*128) into LDS; rows past M and columns past K are
  // zero.  The first batch's loads are issued before the weight ring's, so
  // the ring's prefetch overlaps the staging.
  uint4 xh[XB], xl[XB];
  const int ldx = a.ldx;
  const uint16_t* const X = a.X + (MS ? (size_t)half * MT * 16 * ldx : 0);
#pragma unroll
  for (int q = 0; q < XB; ++q) {
    const int e = threadIdx.x + 256 * q;
    const int m = e / UPR, u = e - m * UPR;
    const int col = k0 + 8 * u;
    const bool ok = m < M && col < K;
    const uint16_t* src = X + (ok ? (size_t)m * ldx + col : 0);
    const uint4 h = *reinterpret_cast<const uint4*>(src);
    const uint4 l = *reinterpret_cast<const uint4*>(src + (ok ? K : 0));
    xh[q] = ok ? h : make_uint4(0, 0, 0, 0);
    xl[q] = ok ? l : make_uint4(0, 0, 0, 0);
  }
  const int wbytes = a.n_tiles * a.nkt * BLOCK_ELEMS * 2;
  const WStream ws1(W, wbytes), ws2(NW == 2 ? W2 : W, wbytes);
  uint4 ring[P][NW][4];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int o = gi * tstride + (kb0 + p) * BLOCK_ELEMS + lane_off;
    const bool in = p < nvb;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int e = in ? o + c * 512 : -1;
      ring[p][0][c] = ws1.load(e);
      if (NW == 2) ring[p][NW - 1][c] = ws2.load(e);
    }
  }
#pragma unroll
  for (int q0 = 0; q0 < NX; q0 += XB) {
    if (q0 > 0) {
#pragma unroll
      for (int q = 0; q < XB; ++q) {
        const int e = threadIdx.x + 256 * (q0 + q);
        const int m = e / UPR, u = e - m * UPR;
        const int col = k0 + 8 * u;
        const bool ok = m < M && col < K;
        const uint16_t* src = X + (ok ? (size_t)m * ldx + col : 0);
        const uint4 h = *reinterpret_cast<const uint4*>(src);
        const uint4 l = *reinterpret_cast<const uint4*>(src + (ok ? K : 0));
        xh[q] = ok ? h : make_uint4(0, 0, 0, 0);
        xl[q] = ok ? l : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int q = 0; q < XB; ++q) {
      const int e = threadIdx.x + 256 * (q0 + q);
      const int m = e / UPR, u = e - m * UPR;
      const int xi = xs_index(m, u, UPR);
      xs[xi] = xh[q];
      xs[LO + xi] = xl[q];
    }
  }
  __syncthreads();

  const int ldp = a.ldp, off2 = a.off2;
  float* const part =
      a.part + (size_t)s * a.part_split + (MS ? (size_t)half * MT * 16 * ldp : 0);
  float* const sink = a.sink + lane * 4;
  for (int j = 0; j < n_my; ++j) {
    const int tile = gi + j * G;
    // the ring's refills for the next tile; after the last tile they read
    // zeros (out-of-range offsets, no memory access)
    const bool more = j + 1 < n_my;
    const int t_base = tile * tstride + kb0 * BLOCK_ELEMS + lane_off;
    const int tn_base = t_base + G * tstride;
    f32x4 acc[NW][MT];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[w][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    // passes of P blocks over the chunk; ring slot r of pass pp holds block
    // pp + r and is refilled with the block P places further
#pragma unroll 1
    for (int pp = 0; pp < NKB; pp += P) {
#pragma unroll
      for (int r = 0; r < P; ++r) {
        const int p = pp + r;
        uint4 fh[MT][4], fl[MT][4];
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int xi = xs_index(t * 16 + i, p * 16 + 4 * g + c, UPR);
            fh[t][c] = xs[xi];
            fl[t][c] = xs[LO + xi];
          }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
#pragma unroll
          for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < MT; ++t)
              acc[w][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  as_bf16x8(ring[r][w][c]), as_bf16x8(fh[t][c]), acc[w][t], 0, 0, 0);
#pragma unroll
          for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < MT; ++t)
              acc[w][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  as_bf16x8(ring[r][w][c]), as_bf16x8(fl[t][c]), acc[w][t], 0, 0, 0);
        }
        // refill: later in this tile, or in the next one
        const int q = p + P;
        const bool next = q >= NKB;
        const int qb = next ? q - NKB : q;  // block of the chunk
        const bool in = (!next || more) && qb < nvb;
        const int o = (next ? tn_base : t_base) + qb * BLOCK_ELEMS;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int e = in ? o + c * 512 : -1;
          ring[r][0][c] = ws1.load(e);
          if (NW == 2) ring[r][NW - 1][c] = ws2.load(e);
        }
      }
    }
    // C layout of the 16x16 MFMA: lane holds column (lane & 15) = row m,
    // register r holds W row 4*(lane/16) + r
    const int n = tile * TILE_ROWS + wave * 16 + 4 * g;
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const int m = t * 16 + i;
        float* dst = m < M ? part + (size_t)m * ldp + w * off2 + n : sink;
        *reinterpret_cast<float4*>(dst) =
            make_float4(acc[w][t][0], acc[w][t][1], acc[w][t][2], acc[w][t][3]);
      }
  }
}

// Units [256 q0, 256 (q0 + XB)) of the X chunk starting at block kb0 (rows
// past M and columns past K are zero): load_x issues the loads, store_x
// writes them to LDS (XOR-swizzled, hi then lo halves).
template <int MT, int NKB, int XB>
MSD_DEV void load_x(uint4 (&xh)[XB], uint4 (&xl)[XB], const uint16_t* X, int ldx, int M, int K,
                    int kb0, int q0) {
  constexpr int UPR = NKB * KB / 8;
  const int k0 = kb0 * KB;
#pragma unroll
  for (int q = 0; q < XB; ++q) {
    const int e = threadIdx.x + 256 * (q0 + q);
    const int m = e / UPR, u = e - m * UPR;
    const int col = k0 + 8 * u;
    const bool ok = m < M && col < K;
    const uint16_t* src = X + (ok ? (size_t)m * ldx + col : 0);
    const uint4 h = *reinterpret_cast<const uint4*>(src);
    const uint4 l = *reinterpret_cast<const uint4*>(src + (ok ? K : 0));
    xh[q] = ok ? h : make_uint4(0, 0, 0, 0);
    xl[q] = ok ? l : make_uint4(0, 0, 0, 0);
  }
}

template <int MT, int NKB, int XB>
MSD_DEV void store_x(uint4* xs, const uint4 (&xh)[XB], const uint4 (&xl)[XB], int q0) {
  constexpr int UPR = NKB * KB / 8;
  constexpr int LO = MT * 16 * UPR;
#pragma unroll
  for (int q = 0; q < XB; ++q) {
    const int e = threadIdx.x + 256 * (q0 + q);
    const int m = e / UPR, u = e - m * UPR;
    const int xi = xs_index(m, u, UPR);
    xs[xi] = xh[q];
    xs[LO + xi] = xl[q];
  }
}

// The same product with two K chunks per workgroup, for 64-row passes (whose
// X chunk fills LDS at 4 blocks) and the widest 32-row ones: each workgroup
// covers chunks 2s and 2s+1
// of NT tiles, so it writes one partial per tile for the pair, half the
// partials (and half the consumer's reads) of one chunk per workgroup.  The
// weight ring runs through the sequence (chunk 0: tiles 0..NT-1, blocks of
// each; then chunk 1 likewise) without a branch on its loads; every tile
// keeps its accumulators across both chunks.  Between the chunks the
// workgroup restages X in LDS; waiting for those loads also waits for the
// ring's, once per workgroup.  Slots for tiles past the workgroup's last and
// blocks past K read zeros.
//
// NC (3 or 4 instead of 2): more K chunks per workgroup, for 64-row passes
// whose partials would otherwise cost more than the extra X restages.
//
// BO (block outer): within each chunk the sequence runs block by block over
// the tiles, so a block's X fragments are read from LDS once for all of the
// workgroup's tiles instead of once per tile.  Every output element sums the
// same products in the same order either way.  It pays at 64 rows, where
// the per-tile fragment reads (eight 16-byte LDS reads per MFMA row tile and
// K step) held the kernel back: 61-row q/k/v 30.5 -> 25.2 us, down
// 30.4 -> 24.9 us, gate+up 44.8 -> 41.5 us (7B-shaped), 64-row down
// 43.8 -> 34.7 us (Qwen-shaped); the fragments' registers make the SwiGLU
// pair spill from four tiles per workgroup on.
template <int MT, int NW, int NKB, int P, int NT, bool BO, int NC = 2>
__global__ __launch_bounds__(256) void k_gemm2(GemmArgs a) {
  static_assert(NKB % P == 0, "ring slots must divide the chunk");
  extern __shared__ uint4 xs[];
  constexpr int UPR = NKB * KB / 8;
  constexpr int LO = MT * 16 * UPR;
  constexpr int SEQ = NC * NT * NKB;  // blocks of the workgroup's sequence
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, g = lane >> 4;
  const int S = a.S, G = a.G, M = a.M, nkt = a.nkt, n_tiles = a.n_tiles;
  const int s = blockIdx.x % S, gi = blockIdx.x / S;
  const int n_my = gi < n_tiles ? min(NT, (n_tiles - gi + G - 1) / G) : 0;
  if (n_my == 0) return;
  const int kb0 = NC * s * NKB;
  const uint16_t* const W = a.W;
  const uint16_t* const W2 = a.W2;
  const size_t lane_off = (size_t)wave * (BLOCK_ELEMS / 4) + lane * 8;
  const int wbytes = a.n_tiles * a.nkt * BLOCK_ELEMS * 2;
  const WStream ws1(W, wbytes), ws2(NW == 2 ? W2 : W, wbytes);
  // element offset of sequence block q, or -1 for zeros; the
  // sequence of chunk half h is tile by tile (q = (h NT + j) NKB + p), or
  // block by block with BO (q = (h NKB + p) NT + j)
  auto block_off = [&](int q) -> long long {
    const int h = q / (NT * NKB);
    const int j = BO ? q % NT : (q / NKB) % NT, p = BO ? (q / NT) % NKB : q % NKB;
    const int kb = kb0 + h * NKB + p;
    if (q >= SEQ || j >= n_my || kb >= nkt) return -1;
    return ((long long)(gi + j * G) * nkt + kb) * BLOCK_ELEMS + (long long)lane_off;
  };
  constexpr int NX = MT * 16 * UPR / 256;  // X units per thread
  static_assert(NX == 16, "X staging assumes 16 units per thread");
  // the first chunk's X loads go out before the ring's, so that its LDS
  // writes wait for them alone
  uint4 xh[NX], xl[NX];
  load_x<MT, NKB, NX>(xh, xl, a.X, a.ldx, M, a.K, kb0, 0);
  uint4 ring[P][NW][4];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const long long o = block_off(p);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int e = o >= 0 ? (int)o + c * 512 : -1;
      ring[p][0][c] = ws1.load(e);
      if (NW == 2) ring[p][NW - 1][c] = ws2.load(e);
    }
  }
  store_x<MT, NKB, NX>(xs, xh, xl, 0);
  __syncthreads();
  f32x4 acc[NT][NW][MT];
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[j][w][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  // the ring slot of sequence block q is q % P whatever the chunk h (a
  // chunk holds NT * NKB blocks, a multiple of P), so the chunk loop of the
  // SwiGLU pair over more than two chunks stays rolled: unrolled, its
  // registers spill (single weights keep it unrolled: 3 us faster on the 7B
  // LM head at 61 rows)
#pragma unroll((NC == 2 || NW == 1) ? NC : 1)
  for (int h = 0; h < NC; ++h) {
    if (h >= 1) {
      // the next X chunk: its loads go out before the barrier (every wave
      // done with the previous chunk), its LDS writes after
      constexpr int XB = NX / 2;
#pragma unroll
      for (int q0 = 0; q0 < NX; q0 += XB) {
        uint4 yh[XB], yl[XB];
        load_x<MT, NKB, XB>(yh, yl, a.X, a.ldx, M, a.K, kb0 + h * NKB, q0);
        if (q0 == 0) lds_barrier();
        store_x<MT, NKB, XB>(xs, yh, yl, q0);
      }
      lds_barrier();
    }
#define MSD_GEMM2_STEP(Q, J, R)                                                               \
  {                                                                                          \
    const int q_ = (Q), j_ = (J), r_ = (R);                                                  \
    _Pragma("unroll") for (int c = 0; c < 4; ++c) {                                          \
      _Pragma("unroll") for (int w = 0; w < NW; ++w)                                         \
      _Pragma("unroll") for (int t = 0; t < MT; ++t)                                         \
        acc[j_][w][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(                             \
            as_bf16x8(ring[r_][w][c]), as_bf16x8(fh[t][c]), acc[j_][w][t], 0, 0, 0);         \
      _Pragma("unroll") for (int w = 0; w < NW; ++w)                                         \
      _Pragma("unroll") for (int t = 0; t < MT; ++t)                                         \
        acc[j_][w][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(                             \
            as_bf16x8(ring[r_][w][c]), as_bf16x8(fl[t][c]), acc[j_][w][t], 0, 0, 0);         \
    }                                                                                        \
    const long long o_ = block_off(q_ + P);                                                  \
    _Pragma("unroll") for (int c = 0; c < 4; ++c) {                                          \
      const int e_ = o_ >= 0 ? (int)o_ + c * 512 : -1;                                       \
      ring[r_][0][c] = ws1.load(e_);                                                         \
      if (NW == 2) ring[r_][NW - 1][c] = ws2.load(e_);                                       \
    }                                                                                        \
  }
#define MSD_GEMM2_FRAGS(PB)                                                                  \
  _Pragma("unroll") for (int t = 0; t < MT; ++t)                                             \
  _Pragma("unroll") for (int c = 0; c < 4; ++c) {                                            \
    const int xi = xs_index(t * 16 + i, (PB) * 16 + 4 * g + c, UPR);                         \
    fh[t][c] = xs[xi];                                                                       \
    fl[t][c] = xs[LO + xi];                                                                  \
  }
    if constexpr (BO) {
#pragma unroll
      for (int p = 0; p < NKB; ++p) {
        uint4 fh[MT][4], fl[MT][4];
        MSD_GEMM2_FRAGS(p)
#pragma unroll
        for (int j = 0; j < NT; ++j) MSD_GEMM2_STEP((h * NKB + p) * NT + j, j, (p * NT + j) % P)
      }
    } else {
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int p = 0; p < NKB; ++p) {
          uint4 fh[MT][4], fl[MT][4];
          MSD_GEMM2_FRAGS(p)
          MSD_GEMM2_STEP((h * NT + j) * NKB + p, j, p % P)
        }
    }
#undef MSD_GEMM2_STEP
#undef MSD_GEMM2_FRAGS
  }
  const int ldp = a.ldp, off2 = a.off2;
  float* const part = a.part + (size_t)s * a.part_split;
  float* const sink = a.sink + lane * 4;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int n = (gi + j * G) * TILE_ROWS + wave * 16 + 4 * g;
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const int m = t * 16 + i;
        float* dst = (m < M && j < n_my) ? part + (size_t)m * ldp + w * off2 + n : sink;
        *reinterpret_cast<float4*>(dst) =
            make_float4(acc[j][w][t][0], acc[j][w][t][1], acc[j][w][t][2], acc[j][w][t][3]);
      }
  }
}

// Full-K variant for the widest single weights at 64 rows (LM heads of large
// vocabularies, many tiles per workgroup): every workgroup covers all of K
// for NT tiles, chunk by chunk, restaging X in LDS at each chunk and keeping
// the tiles' accumulators in registers throughout.  It writes one partial
// per tile (S = 1), where the chunked kernels write one per K chunk: at the
// Qwen2.5-VL-7B-shaped LM head that is 39 MB instead of 272 MB per 64 rows,
// and as much less for the consumer to read.
//
// With ten tiles' accumulators the X fragments of a whole block no longer
// fit beside them, so a block is taken in two halves of its K steps (MFMA
// steps c = 0, 1 and c = 2, 3), and the register ring holds half blocks:
// 2P of them, as many bytes in flight as P whole blocks.  The ring runs
// half by half over the tiles, q = ((c NKB + p) 2 + hf) NT + j, so one half's
// fragments are read from LDS once for all NT tiles; 2 NKB NT is a multiple
// of 2P, so every chunk uses the same ring slots.  A half block is two
// 1 KB contiguous loads per wave.  Each restage waits for the ring's loads
// in flight (loads complete in order), once per chunk.
template <int MT, int NKB, int P, int NT>
__global__ __launch_bounds__(256) void k_gemm_fk(GemmArgs a) {
  constexpr int PH = 2 * P;           // half-block ring slots
  constexpr int CSEQ = 2 * NKB * NT;  // half blocks per chunk
  static_assert(CSEQ % PH == 0, "every chunk must start at ring slot 0");
  extern __shared__ uint4 xs[];
  constexpr int UPR = NKB * KB / 8;
  constexpr int LO = MT * 16 * UPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, g = lane >> 4;
  const int G = a.G, M = a.M, nkt = a.nkt, n_tiles = a.n_tiles;
  const int gi = blockIdx.x;
  const int n_my = gi < n_tiles ? min(NT, (n_tiles - gi + G - 1) / G) : 0;
  if (n_my == 0) return;
  const int n_ch = (nkt + NKB - 1) / NKB;
  const uint16_t* const W = a.W;
  const size_t lane_off = (size_t)wave * (BLOCK_ELEMS / 4) + lane * 8;
  // element offset of sequence half block q, or -1 for zeros
  const WStream ws1(W, a.n_tiles * a.nkt * BLOCK_ELEMS * 2);
  auto half_off = [&](int q) -> long long {
    const int c = q / CSEQ, r = q - c * CSEQ;
    const int ph = r / NT, j = r - ph * NT;
    const int kb = c * NKB + (ph >> 1);
    if (j >= n_my || kb >= nkt) return -1;
    return ((long long)(gi + j * G) * nkt + kb) * BLOCK_ELEMS + (long long)lane_off +
           (ph & 1) * 1024;
  };
  constexpr int NX = MT * 16 * UPR / 256;
  static_assert(NX == 16, "X staging assumes 16 units per thread");
  uint4 xh[NX], xl[NX];
  load_x<MT, NKB, NX>(xh, xl, a.X, a.ldx, M, a.K, 0, 0);
  uint4 ring[PH][2];
#pragma unroll
  for (int q = 0; q < PH; ++q) {
    const long long o = half_off(q);
    ring[q][0] = ws1.load((int)o);
    ring[q][1] = ws1.load(o >= 0 ? (int)o + 512 : -1);
  }
  store_x<MT, NKB, NX>(xs, xh, xl, 0);
  __syncthreads();
  f32x4 acc[NT][MT];
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
  for (int ch = 0; ch < n_ch; ++ch) {
    if (ch > 0) {
      // the chunk's X: loads before the barrier (every wave done with the
      // previous chunk), LDS writes after
      constexpr int XB = NX / 2;
#pragma unroll
      for (int q0 = 0; q0 < NX; q0 += XB) {
        uint4 yh[XB], yl[XB];
        load_x<MT, NKB, XB>(yh, yl, a.X, a.ldx, M, a.K, ch * NKB, q0);
        if (q0 == 0) lds_barrier();
        store_x<MT, NKB, XB>(xs, yh, yl, q0);
      }
      lds_barrier();
    }
#pragma unroll
    for (int ph = 0; ph < 2 * NKB; ++ph) {
      const int p = ph >> 1, hf = ph & 1;
      uint4 fh[MT][2], fl[MT][2];
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int xi = xs_index(t * 16 + i, p * 16 + 4 * g + 2 * hf + c, UPR);
          fh[t][c] = xs[xi];
          fl[t][c] = xs[LO + xi];
        }
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int r = (ph * NT + j) % PH;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
#pragma unroll
          for (int t = 0; t < MT; ++t)
            acc[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                as_bf16x8(ring[r][c]), as_bf16x8(fh[t][c]), acc[j][t], 0, 0, 0);
#pragma unroll
          for (int t = 0; t < MT; ++t)
            acc[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                as_bf16x8(ring[r][c]), as_bf16x8(fl[t][c]), acc[j][t], 0, 0, 0);
        }
        const long long o = half_off(ch * CSEQ + ph * NT + j + PH);
        ring[r][0] = ws1.load((int)o);
        ring[r][1] = ws1.load(o >= 0 ? (int)o + 512 : -1);
      }
    }
  }
  const int ldp = a.ldp;
  float* const part = a.part;
  float* const sink = a.sink + lane * 4;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int n = (gi + j * G) * TILE_ROWS + wave * 16 + 4 * g;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int m = t * 16 + i;
      float* dst = (m < M && j < n_my) ? part + (size_t)m * ldp + n : sink;
      *reinterpret_cast<float4*>(dst) =
          make_float4(acc[j][t][0], acc[j][t][1], acc[j][t][2], acc[j][t][3]);
    }
  }
}

// One thread per 16-byte unit of the packed layout.
__global__ void k_pack(const uint16_t* src, int N, int K, int nkt, size_t units, uint16_t* dst) {
  const size_t q = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= units) return;
  const int lane = (int)(q & 63);
  const size_t r = q >> 6;  // (t * nkt + kb) * 16 + wave * 4 + c
  const int c = (int)(r & 3), wave = (int)((r >> 2) & 3);
  const size_t blk = r >> 4;
  const int kb = (int)(blk % nkt);
  const int t = (int)(blk / nkt);
  const int row = t * TILE_ROWS + wave * 16 + (lane & 15);
  const int col = kb * KB + 32 * (lane >> 4) + 8 * c;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (row < N && col < K) v = *reinterpret_cast<const uint4*>(src + (size_t)row * K + col);
  *reinterpret_cast<uint4*>(dst + q * 8) = v;
}

// The inverse of k_pack: row-major bf16 [N][K] from the packed layout.
__global__ void k_unpack(const uint16_t* src, int N, int K, int nkt, size_t units, uint16_t* dst) {
  const size_t q = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= units) return;
  const int lane = (int)(q & 63);
  const size_t r = q >> 6;
  const int c = (int)(r & 3), wave = (int)((r >> 2) & 3);
  const size_t blk = r >> 4;
  const int kb = (int)(blk % nkt);
  const int t = (int)(blk / nkt);
  const int row = t * TILE_ROWS + wave * 16 + (lane & 15);
  const int col = kb * KB + 32 * (lane >> 4) + 8 * c;
  if (row < N && col < K)
    *reinterpret_cast<uint4*>(dst + (size_t)row * K + col) =
        *reinterpret_cast<const uint4*>(src + q * 8);
}

// With timing events the launch carries them in its dispatch packet, so they
// bracket the kernel's execution only.
template <int MT, int NW>
void launch_mt(dim3 grid, const GemmArgs& a, const GemmScratch& sc, hipStream_t st) {
  constexpr int P = RING;
  constexpr int NKB = chunk_blocks(MT);
  const size_t lds = (size_t)MT * 16 * NKB * KB * 4;
  if (sc.ev_start)
    hipExtLaunchKernelGGL((k_gemm<MT, NW, NKB, P>), grid, dim3(256), lds, st, sc.ev_start,
                          sc.ev_stop, 0, a);
  else
    hipLaunchKernelGGL((k_gemm<MT, NW, NKB, P>), grid, dim3(256), lds, st, a);
}

template <int MT, int NW, int NT, int NC = 2>
void launch_pair(dim3 grid, const GemmArgs& a, const GemmScratch& sc, hipStream_t st) {
  constexpr int P = RING;
  constexpr int NKB = chunk_blocks(MT);
  // block outer at 64 rows, but for the SwiGLU pair from four tiles on
  constexpr bool BO = MT == 4 && (NW == 1 || NT <= 3);
  const size_t lds = (size_t)MT * 16 * NKB * KB * 4;
  if (sc.ev_start)
    hipExtLaunchKernelGGL((k_gemm2<MT, NW, NKB, P, NT, BO, NC>), grid, dim3(256), lds, st,
                          sc.ev_start, sc.ev_stop, 0, a);
  else
    hipLaunchKernelGGL((k_gemm2<MT, NW, NKB, P, NT, BO, NC>), grid, dim3(256), lds, st, a);
}

template <int NT>
void launch_fk(dim3 grid, const GemmArgs& a, const GemmScratch& sc, hipStream_t st) {
  constexpr int MT = 4, P = RING;
  constexpr int NKB = chunk_blocks(MT);
  const size_t lds = (size_t)MT * 16 * NKB * KB * 4;
  if (sc.ev_start)
    hipExtLaunchKernelGGL((k_gemm_fk<MT, NKB, P, NT>), grid, dim3(256), lds, st, sc.ev_start,
                          sc.ev_stop, 0, a);
  else
    hipLaunchKernelGGL((k_gemm_fk<MT, NKB, P, NT>), grid, dim3(256), lds, st, a);
}

// The SwiGLU pair over more than two chunks takes at most four tiles per
// workgroup (PAIR_NC_MAX_TILES): at five its registers spill.
constexpr int PAIR_NC_MAX_TILES = 4;
template <int MT, int NW, int NC = 2>
void launch_pair_nt(int nt, dim3 grid, const GemmArgs& a, const GemmScratch& sc, hipStream_t st) {
  if (nt == 1) launch_pair<MT, NW, 1, NC>(grid, a, sc, st);
  else if (nt == 2) launch_pair<MT, NW, 2, NC>(grid, a, sc, st);
  else if (nt == 3) launch_pair<MT, NW, 3, NC>(grid, a, sc, st);
  else if (nt == 4) launch_pair<MT, NW, 4, NC>(grid, a, sc, st);
  else if constexpr (NW == 1 || NC == 2) launch_pair<MT, NW, 5, NC>(grid, a, sc, st);
}

// Streaming read of a buffer with the weight stream's access pattern: every
// wave instruction reads 1 KB contiguous with nontemporal loads, four in
// flight per lane per step, workgroups striding over 64 KB spans.  The XOR
// of everything read keeps the loads alive; a workgroup writes one word only
// if it equals a value the data never produce here (zero-filled buffers).
__global__ __launch_bounds__(256) void k_stream_read(const uint16_t* buf, size_t spans,
                                                     unsigned* sink) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint4 acc = make_uint4(0, 0, 0, 0);
  for (size_t sp = blockIdx.x; sp < spans; sp += gridDim.x) {
    const uint16_t* b = buf + sp * (size_t)(4 * BLOCK_ELEMS) + (size_t)wave * (BLOCK_ELEMS / 4) +
                        lane * 8;
    uint4 v[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q] = load_stream(b + (q / 4) * BLOCK_ELEMS + (q % 4) * 512);
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      acc.x ^= v[q].x;
      acc.y ^= v[q].y;
      acc.z ^= v[q].z;
      acc.w ^= v[q].w;
    }
  }
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9E3779B9u) sink[blockIdx.x] = 1u;
}

}  // namespace

size_t stream_span_bytes() { return (size_t)4 * BLOCK_ELEMS * sizeof(uint16_t); }

void launch_stream_read(const uint16_t* buf, size_t spans, int wgs, unsigned* sink,
                        hipStream_t st) {
  hipLaunchKernelGGL(k_stream_read, dim3(wgs), dim3(256), 0, st, buf, spans, sink);
}

void launch_unpack(const uint16_t* src, int N, int K, uint16_t* dst, hipStream_t st) {
  const int nkt = (K + KB - 1) / KB;
  const size_t units = packed_elems(N, K) / 8;
  hipLaunchKernelGGL(k_unpack, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, st, src, N, K,
                     nkt, units, dst);
}

size_t packed_elems(int N, int K) {
  return (size_t)((N + TILE_ROWS - 1) / TILE_ROWS) * ((K + KB - 1) / KB) * BLOCK_ELEMS;
}

void launch_pack(const uint16_t* src, int N, int K, uint16_t* dst, hipStream_t st) {
  const int nkt = (K + KB - 1) / KB;
  const size_t units = packed_elems(N, K) / 8;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, st, src, N, K,
                     nkt, units, dst);
}

GemmPlan plan_gemm(int M, int N, int K, int nw, int target_wgs) {
  GemmPlan p;
  const int mc = M < 64 ? M : 64;
  p.MT = mc <= 16 ? 1 : (mc <= 32 ? 2 : 4);
  p.nkt = (K + KB - 1) / KB;
  p.nkb = chunk_blocks(p.MT);
  p.S = (p.nkt + p.nkb - 1) / p.nkb;
  p.n_tiles = (N + TILE_ROWS - 1) / TILE_ROWS;
  // workgroups per chunk: about target_wgs in total, every workgroup of a
  // chunk getting the same number of tiles
  int G = (target_wgs + p.S - 1) / p.S;
  if (G > p.n_tiles) G = p.n_tiles;
  if (G < 1) G = 1;
  int per = (p.n_tiles + G - 1) / G;
  G = (p.n_tiles + per - 1) / per;
  // one workgroup per CU: a few workgroups past the target would run as a
  // second wave, so take more tiles per workgroup instead
  while (p.S * G > target_wgs && G > 1) {
    ++per;
    G = (p.n_tiles + per - 1) / per;
  }
  p.G = G;
  p.pair = 0;
  p.per = per;
  // Two K chunks per workgroup (the tiles' accumulators live in registers,
  // at most PAIR_MAX_TILES of them).  64-row passes: when at least three
  // quarters of the target workgroups stay busy.  32-row passes, whose
  // partials are half as many per weight byte: the SwiGLU pair always (its
  // 9.5 MB of partials at the 7B shape cost more than the idle CUs: gate+up
  // 37.0 -> 36.1 us, its consumer about 1 us less), single weights only when
  // the workgroup count stays within 5% and each workgroup has four tiles or
  // more to amortise the mid-stream restage of X (the wide LM heads).
  if ((p.MT == 4 || p.MT == 2) && p.S >= 2) {
    const int S2 = (p.S + 1) / 2;
    int G2 = (target_wgs + S2 - 1) / S2;
    if (G2 > p.n_tiles) G2 = p.n_tiles;
    int per2 = (p.n_tiles + G2 - 1) / G2;
    G2 = (p.n_tiles + per2 - 1) / per2;
    while (S2 * G2 > target_wgs && G2 > 1) {
      ++per2;
      G2 = (p.n_tiles + per2 - 1) / per2;
    }
    const bool busy = p.MT == 4 ? 4 * S2 * G2 >= 3 * target_wgs
                                : (nw == 2 || (per2 >= 4 && 20 * S2 * G2 >= 19 * p.S * p.G));
    if (per2 <= PAIR_MAX_TILES && busy) {
      p.pair = 2;
      p.S = S2;
      p.G = G2;
      p.per = per2;
    }
  }
  // Full K per workgroup for the widest single weights at 64 rows: when
  // every workgroup would take FK_MIN_TILES tiles or more at one chunk each,
  // the X restage per chunk costs less than the chunk partials it saves
  p.fk = 0;
  if (p.MT == 4 && nw == 1) {
    int nt = (p.n_tiles + target_wgs - 1) / target_wgs;
    nt = (nt + 1) / 2 * 2;  // launched tile counts are even
    if (nt >= FK_MIN_TILES && nt <= FK_MAX_TILES) {
      p.fk = nt;
      p.pair = 0;
      p.S = 1;
      p.G = (p.n_tiles + nt - 1) / nt;
      p.per = nt;
    }
  }
  p.nw = nw;
  p.ldp = p.n_tiles * TILE_ROWS * nw;
  p.off2 = p.n_tiles * TILE_ROWS;
  p.ms = 0;
  // 33-64 rows, single weights with at most two tiles per workgroup: the X
  // chunk costs as much as the weight blocks streamed against it, so the
  // pass runs as two 32-row halves with 8-block chunks (each workgroup
  // streaming twice the weight bytes per X byte; the output projection at
  // 61 rows 14.7 -> 12.0 us, Qwen2.5-VL-7B-shaped).  Wider weights stay
  // whole: there the doubled weight stream per CU (the partner's blocks are
  // L2 hits, but they still pass through the CU) costs more than the
  // halved partials save.
  if (p.MT == 4 && nw == 1 && !p.fk && p.per <= 2) {
    const GemmPlan h = plan_gemm(32, N, K, nw, target_wgs / 2);
    if (!h.pair && !h.fk) {
      p = h;  // same ldp and off2: they depend on N and nw only
      p.ms = 1;
    }
  }
  // 64-row passes: four or three K chunks per workgroup where that writes
  // fewer partials.  Single weights: on about as many workgroups, each with
  // four tiles or more to amortise the X restage between chunks (the 7B LM
  // head at 61 rows: 8 -> 2 partials, 66.6 -> 55.9 us); not with fewer
  // tiles (7B down on 256 workgroups of two tiles: 24.9 -> 26.8 us) or
  // fewer workgroups (7B q/k/v 27.2 -> 31.0 us on 192 instead of 256).  The
  // SwiGLU pair: while three quarters of the target workgroups stay busy,
  // since its consumer reads every partial of both weights (Qwen-shaped
  // 61-row verify 4.71 -> 4.59 ms with 2 partials instead of 4).
  if (p.MT == 4 && !p.fk && !p.ms) {
    const int S1 = (p.nkt + p.nkb - 1) / p.nkb;
    for (int nc = 4; nc >= 3; --nc) {
      const int Sn = (S1 + nc - 1) / nc;
      if (Sn >= p.S) continue;
      int Gn = (target_wgs + Sn - 1) / Sn;
      if (Gn > p.n_tiles) Gn = p.n_tiles;
      int pern = (p.n_tiles + Gn - 1) / Gn;
      Gn = (p.n_tiles + pern - 1) / pern;
      while (Sn * Gn > target_wgs && Gn > 1) {
        ++pern;
        Gn = (p.n_tiles + pern - 1) / pern;
      }
      const bool keep = nw == 2 ? 4 * Sn * Gn >= 3 * target_wgs : 20 * Sn * Gn >= 19 * p.S * p.G;
      const int max_tiles = nw == 2 ? PAIR_NC_MAX_TILES : PAIR_MAX_TILES;
      if ((nw == 2 || pern >= 4) && pern <= max_tiles && keep) {
        p.pair = nc;
        p.S = Sn;
        p.G = Gn;
        p.per = pern;
        break;
      }
    }
  }
  return p;
}

size_t gemm_part_floats(int M, int N, int K, int nw, int target_wgs) {
  const GemmPlan p = plan_gemm(M, N, K, nw, target_wgs);
  return (size_t)p.S * M * p.ldp;
}

void launch_gemm(const uint16_t* X, int ldx, int M, const uint16_t* W, const uint16_t* W2, int N,
                 int K, float* part, float* sink, const GemmScratch& sc,
                 hipStream_t st) {
  const int nw = W2 ? 2 : 1;
  const GemmPlan pl = plan_gemm(M, N, K, nw, sc.target_wgs);
  GemmArgs a{};
  a.X = X;
  a.ldx = ldx;
  a.M = M;
  a.K = K;
  a.W = W;
  a.W2 = W2;
  a.n_tiles = pl.n_tiles;
  a.nkt = pl.nkt;
  a.S = pl.S;
  a.G = pl.G;
  a.part = part;
  a.part_split = (size_t)M * pl.ldp;
  a.ldp = pl.ldp;
  a.off2 = pl.off2;
  a.sink = sink;
  if (pl.ms) {
    const dim3 grid(16 * ((pl.S * pl.G + 7) / 8));
    constexpr int NKB = chunk_blocks(2);
    const size_t lds = (size_t)2 * 16 * NKB * KB * 4;
    if (sc.ev_start)
      hipExtLaunchKernelGGL((k_gemm<2, 1, NKB, RING, true>), grid, dim3(256), lds, st, sc.ev_start,
                            sc.ev_stop, 0, a);
    else
      hipLaunchKernelGGL((k_gemm<2, 1, NKB, RING, true>), grid, dim3(256), lds, st, a);
    return;
  }
  const dim3 grid(pl.S * pl.G);
  if (pl.fk) {
    if (pl.fk == 8) launch_fk<8>(grid, a, sc, st);
    else launch_fk<10>(grid, a, sc, st);
    return;
  }
  if (pl.pair == 4) {
    if (nw == 2) launch_pair_nt<4, 2, 4>(pl.per, grid, a, sc, st);
    else launch_pair_nt<4, 1, 4>(pl.per, grid, a, sc, st);
    return;
  }
  if (pl.pair == 3) {
    if (nw == 2) launch_pair_nt<4, 2, 3>(pl.per, grid, a, sc, st);
    else launch_pair_nt<4, 1, 3>(pl.per, grid, a, sc, st);
    return;
  }
  if (pl.pair == 2) {
    if (pl.MT == 2 && nw == 2) launch_pair_nt<2, 2>(pl.per, grid, a, sc, st);
    else if (pl.MT == 2) launch_pair_nt<2, 1>(pl.per, grid, a, sc, st);
    else if (nw == 2) launch_pair_nt<4, 2>(pl.per, grid, a, sc, st);
    else launch_pair_nt<4, 1>(pl.per, grid, a, sc, st);
    return;
  }
  if (nw == 2) {
    if (pl.MT == 1) launch_mt<1, 2>(grid, a, sc, st);
    else if (pl.MT == 2) launch_mt<2, 2>(grid, a, sc, st);
    else launch_mt<4, 2>(grid, a, sc, st);
  } else {
    if (pl.MT == 1) launch_mt<1, 1>(grid, a, sc, st);
    else if (pl.MT == 2) launch_mt<2, 1>(grid, a, sc, st);
    else launch_mt<4, 1>(grid, a, sc, st);
  }
}

}  // namespace msd
