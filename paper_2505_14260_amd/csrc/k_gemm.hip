// Thin-M GEMM on gfx950 MFMA: P_s[m][n] = sum_{k in chunk s} X[m][k] * W[n][k],
// W in bfloat16, X as split rows (bf16 hi + lo).
//
// The decode path multiplies a few dozen activation rows (tree nodes) by
// large weight matrices, so the kernel is bound by streaming W from HBM once.
// Layout of the work:
//  - K is cut into S chunks.  A workgroup (4 waves) owns one chunk s and a
//    strided set of 64-row tiles of W (and of W2 for the SwiGLU pair); it
//    stages its X chunk into LDS once and then streams the W rows of all its
//    tiles, each wave owning 16 rows of a tile, with a ring of P register
//    stages whose prefetch runs across tile boundaries.  No workgroup or wave
//    ever waits for another one.
//  - X arrives split by its producer, x = hi + lo with hi = bf16(x) and
//    lo = bf16(x - hi), so W x = W hi + W lo carries about 16 significant bits
//    of the activations (one bf16 rounding of every GEMM input, amplified by
//    a deep stack of layers, is far larger than the error of the weights'
//    products themselves).  Two MFMAs per step; the kernel stays bound by
//    the weight stream.
//  - v_mfma_f32_16x16x32_bf16 with A = W rows (from HBM) and B = X^T (from
//    LDS).  The K index inside one MFMA may be any permutation shared by A and
//    B, so a lane loads 32 physically contiguous bf16 of its W row (the four
//    lanes of a row cover 256 contiguous bytes per block).
//  - Each chunk's partial product is stored in float32 as part[s][m][n]; the
//    kernel that consumes the product (residual + RMSNorm, RoPE + KV write,
//    SwiGLU, vocabulary top-k) sums the S partials in chunk order, so the
//    result is deterministic.
#include <hip/hip_ext.h>

#include "msd_internal.h"

namespace msd {

namespace {

constexpr int KB = 128;  // K elements per block
constexpr int WAVES = 4;
constexpr int TILE_ROWS = 16 * WAVES;

template <int NW>
struct WFrag {
  uint4 w[NW][4];
};

// W block load for one lane: 32 contiguous bf16 of its row starting at k.
// TAIL: the chunk may end inside the block; columns past kend read a clamped
// address and are zeroed.
template <int NW, bool TAIL>
MSD_DEV void load_w(WFrag<NW>& f, const uint16_t* const (&wrow)[NW], int k, int kend) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int kk = k + 8 * c;
    const bool ok = !TAIL || kk < kend;
    const int kc = ok ? kk : kend - 8;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint4 v = *reinterpret_cast<const uint4*>(wrow[w] + kc);
      f.w[w][c] = ok ? v : make_uint4(0, 0, 0, 0);
    }
  }
}

// LDS X chunk: row m holds the chunk's columns in 16-byte units (8 bf16);
// unit u of row m is stored at u ^ (m & 15) so that the 16 rows read by one
// MFMA operand load hit different banks.  The lo halves follow the hi halves.
MSD_DEV int xs_index(int m, int u, int units_per_row) { return m * units_per_row + (u ^ (m & 15)); }

// Row pointers of W (and W2) for 16-row group `row0` of a tile; only
// constant indices into the argument block are used: a runtime index would
// become a memory load whose wait drains every outstanding weight load.
template <int NW>
MSD_DEV void row_ptrs(const uint16_t* (&wrow)[NW], int n, int N, int K, const uint16_t* w0,
                      const uint16_t* w1, const uint16_t* w2, int e0, int e1,
                      const uint16_t* wb2) {
  const int nn = n < N ? n : 0;
  const uint16_t* wb = nn < e0 ? w0 : (nn < e1 ? w1 : w2);
  const int base = nn < e0 ? 0 : (nn < e1 ? e0 : e1);
  wrow[0] = wb + (size_t)(nn - base) * K;
  if (NW == 2) wrow[NW - 1] = wb2 + (size_t)nn * K;
}

template <int MT, int NW, int P, bool TAIL>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  extern __shared__ uint4 xs[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i = lane & 15, g = lane >> 4;
  // scalar copies of the arguments
  const int N = a.N, K = a.K, M = a.M, G = a.G, S = a.S, Kc = a.Kc;
  const uint16_t* const w0 = a.Wseg[0];
  const uint16_t* const w1 = a.Wseg[1];
  const uint16_t* const w2 = a.Wseg[2];
  const uint16_t* const wb2 = a.W2;
  const int e0 = a.seg_end[0], e1 = a.seg_end[1];
  float* const part = a.part;
  const size_t part_split = a.part_split;
  const int ldp = a.ldp;

  const int s = blockIdx.x % S;
  const int gi = blockIdx.x / S;
  const int k0 = s * Kc;
  const int kend = min(K, k0 + Kc);
  const int nkb = (kend - k0 + KB - 1) / KB;
  const int upr = Kc / 8;  // 16-byte units per LDS row
  const int n_tiles = (N + TILE_ROWS - 1) / TILE_ROWS;
  const int n_my = gi < n_tiles ? (n_tiles - gi + G - 1) / G : 0;
  const int total = n_my * nkb;
  const int row_in_tile = wave * 16 + i;

  // stage X[0:MT*16, k0:k0+nkb*128) into LDS (rows past M and columns past
  // kend are zero).  Issued before the weight prefetch: loads complete in
  // order, so staging first does not wait for the first weight blocks.
  const int units = nkb * (KB / 8);
  const int lo_base = MT * 16 * upr;
  for (int e = threadIdx.x; e < MT * 16 * units; e += 256) {
    const int m = e / units, u = e - m * units;
    const int col = k0 + 8 * u;
    uint4 hi = make_uint4(0, 0, 0, 0), lo = hi;
    if (m < M && col < kend) {
      const uint16_t* src = a.X + (size_t)m * a.ldx + col;
      hi = *reinterpret_cast<const uint4*>(src);
      lo = *reinterpret_cast<const uint4*>(src + K);
    }
    const int xi = xs_index(m, u, upr);
    xs[xi] = hi;
    xs[lo_base + xi] = lo;
  }
  WFrag<NW> ring[P];
  if (total > 0) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int f = min(p, total - 1);
      const uint16_t* wr[NW];
      row_ptrs<NW>(wr, (gi + (f / nkb) * G) * TILE_ROWS + row_in_tile, N, K, w0, w1, w2, e0, e1,
                   wb2);
      load_w<NW, TAIL>(ring[p], wr, k0 + (f % nkb) * KB + 32 * g, kend);
    }
  }

  __syncthreads();
  if (total == 0) return;

  f32x4 acc[NW][MT];
#pragma unroll
  for (int w = 0; w < NW; ++w)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[w][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // flattened (tile, block) sequence; the prefetch index is clamped, and a
  // tile's partial is stored after its last block
  for (int f0 = 0; f0 < total; f0 += P) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int f = f0 + p;
      if (f < total) {
        const int kb = f % nkb;
        uint4 xh[MT][4], xl[MT][4];
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int xi = xs_index(t * 16 + i, kb * 16 + 4 * g + c, upr);
            xh[t][c] = xs[xi];
            xl[t][c] = xs[lo_base + xi];
          }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
#pragma unroll
          for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < MT; ++t)
              acc[w][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  as_bf16x8(ring[p].w[w][c]), as_bf16x8(xh[t][c]), acc[w][t], 0, 0, 0);
#pragma unroll
          for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < MT; ++t)
              acc[w][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  as_bf16x8(ring[p].w[w][c]), as_bf16x8(xl[t][c]), acc[w][t], 0, 0, 0);
        }
        const int fn = min(f + P, total - 1);
        const uint16_t* wr[NW];
        row_ptrs<NW>(wr, (gi + (fn / nkb) * G) * TILE_ROWS + row_in_tile, N, K, w0, w1, w2, e0, e1,
                     wb2);
        load_w<NW, TAIL>(ring[p], wr, k0 + (fn % nkb) * KB + 32 * g, kend);
        if (kb == nkb - 1) {
          // C layout of the 16x16 MFMA: lane holds column (lane & 15) = row
          // m, register r holds W row 4*(lane/16) + r
          const int n = (gi + (f / nkb) * G) * TILE_ROWS + wave * 16 + 4 * g;
#pragma unroll
          for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < MT; ++t) {
              const int m = t * 16 + i;
              if (m < M && n < N) {
                float* dst = part + (size_t)s * part_split + (size_t)m * ldp + w * N + n;
                *reinterpret_cast<float4*>(dst) =
                    make_float4(acc[w][t][0], acc[w][t][1], acc[w][t][2], acc[w][t][3]);
              }
              acc[w][t] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
        }
      }
    }
  }
}

// With timing events the launch carries them in its dispatch packet, so they
// bracket the kernel's execution only.
template <int MT, int NW, bool TAIL>
void launch_one(dim3 grid, size_t lds, const GemmArgs& a, const GemmScratch& sc,
                hipStream_t st) {
  constexpr int P = NW == 2 ? 3 : 4;
  if (sc.ev_start)
    hipExtLaunchKernelGGL((k_gemm<MT, NW, P, TAIL>), grid, dim3(256), lds, st, sc.ev_start,
                          sc.ev_stop, 0, a);
  else
    hipLaunchKernelGGL((k_gemm<MT, NW, P, TAIL>), grid, dim3(256), lds, st, a);
}

template <int MT>
void launch_mt(int nw, bool tail, dim3 grid, size_t lds, const GemmArgs& a,
               const GemmScratch& sc, hipStream_t st) {
  if (nw == 2) {
    if (tail) launch_one<MT, 2, true>(grid, lds, a, sc, st);
    else launch_one<MT, 2, false>(grid, lds, a, sc, st);
  } else {
    if (tail) launch_one<MT, 1, true>(grid, lds, a, sc, st);
    else launch_one<MT, 1, false>(grid, lds, a, sc, st);
  }
}

}  // namespace

GemmPlan plan_gemm(int M, int N, int K, int nw, int target_wgs, int lds_bytes) {
  GemmPlan p;
  const int mc = M < 64 ? M : 64;
  p.MT = mc <= 16 ? 1 : (mc <= 32 ? 2 : 4);
  // X chunk in LDS: MT*16 rows of Kc bf16 pairs (hi, lo) within lds_bytes
  const int kc_max = (lds_bytes / 4 / (p.MT * 16)) / KB * KB;
  p.S = (K + kc_max - 1) / kc_max;
  p.Kc = ((K + p.S - 1) / p.S + KB - 1) / KB * KB;
  p.S = (K + p.Kc - 1) / p.Kc;
  // workgroups per chunk: about target_wgs in total, with every workgroup
  // of a chunk getting the same number of tiles
  const int n_tiles = (N + TILE_ROWS - 1) / TILE_ROWS;
  int G = (target_wgs + p.S - 1) / p.S;
  if (G > n_tiles) G = n_tiles;
  if (G < 1) G = 1;
  const int per = (n_tiles + G - 1) / G;
  p.G = (n_tiles + per - 1) / per;
  p.nw = nw;
  return p;
}

size_t gemm_part_floats(int M, int N, int K, int nw, int target_wgs, int lds_bytes) {
  const GemmPlan p = plan_gemm(M, N, K, nw, target_wgs, lds_bytes);
  return (size_t)p.S * M * N * nw;
}

void launch_gemm(const uint16_t* X, int ldx, int M, const uint16_t* const* Wseg,
                 const int* seg_rows, int n_seg, const uint16_t* W2, int K, float* part,
                 const GemmScratch& sc, hipStream_t st) {
  int N = 0;
  GemmArgs base{};
  for (int q = 0; q < 3; ++q) {
    if (q < n_seg) {
      N += seg_rows[q];
      base.Wseg[q] = Wseg[q];
    } else {
      base.Wseg[q] = Wseg[0];
    }
    base.seg_end[q] = N;
  }
  const int nw = W2 ? 2 : 1;
  const GemmPlan pl = plan_gemm(M, N, K, nw, sc.target_wgs, sc.lds_bytes);
  // chunks are whole 128-column blocks except when K itself is not
  const bool tail = (K % KB) != 0;
  const size_t lds = (size_t)pl.MT * 16 * pl.Kc * 4;
  GemmArgs a = base;
  a.X = X;
  a.ldx = ldx;
  a.M = M;
  a.W2 = W2;
  a.N = N;
  a.K = K;
  a.S = pl.S;
  a.Kc = pl.Kc;
  a.G = pl.G;
  a.ldp = N * nw;
  a.part_split = (size_t)M * N * nw;
  a.part = part;
  dim3 grid(pl.S * pl.G);
  if (pl.MT == 1) launch_mt<1>(nw, tail, grid, lds, a, sc, st);
  else if (pl.MT == 2) launch_mt<2>(nw, tail, grid, lds, a, sc, st);
  else launch_mt<4>(nw, tail, grid, lds, a, sc, st);
}

}  // namespace msd
