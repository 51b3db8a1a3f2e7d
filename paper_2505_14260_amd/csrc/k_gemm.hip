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
// 64 KB spans, read with nontemporal loads.  Within one MFMA the K index may
// be any permutation shared by the two operands; the X fragments use the
// same permutation.
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

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
MSD_DEV uint4 load_stream(const uint16_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// LDS X chunk: row m holds the chunk's columns in 16-byte units (8 bf16);
// unit u of row m is stored at u ^ (m & 15) so that the 16 rows read by one
// MFMA operand load hit different banks.
MSD_DEV int xs_index(int m, int u, int upr) { return m * upr + (u ^ (m & 15)); }

template <int MT, int NW, int NKB, int P>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  static_assert(NKB % P == 0, "ring slots must divide the chunk");
  extern __shared__ uint4 xs[];
  constexpr int UPR = NKB * KB / 8;  // 16-byte units per LDS row
  constexpr int LO = MT * 16 * UPR;  // offset of the lo halves
  constexpr int NX = MT * 16 * UPR / 256;
  constexpr int XB = NX < 16 ? NX : 16;  // staging batch (loads in flight)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, g = lane >> 4;
  const int S = a.S, G = a.G, K = a.K, M = a.M, nkt = a.nkt, n_tiles = a.n_tiles;
  const int s = blockIdx.x % S, gi = blockIdx.x / S;
  const int n_my = gi < n_tiles ? (n_tiles - gi + G - 1) / G : 0;
  if (n_my == 0) return;
  const int kb0 = s * NKB;
  const int k0 = kb0 * KB;
  const uint16_t* const W = a.W;
  const uint16_t* const W2 = a.W2;
  const size_t lane_off = (size_t)wave * (BLOCK_ELEMS / 4) + lane * 8;
  const size_t tstride = (size_t)nkt * BLOCK_ELEMS;
  // the chunk's blocks; past K (last chunk) the loads read the zero block,
  // X being zero there too
  const int nvb = min(NKB, nkt - kb0);

  // X[0:MT*16, k0:k0+NKB*128) into LDS; rows past M and columns past K are
  // zero.  The first batch's loads are issued before the weight ring's, so
  // the ring's prefetch overlaps the staging.
  uint4 xh[XB], xl[XB];
  const uint16_t* const X = a.X;
  const int ldx = a.ldx;
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
  const uint16_t* const dummy = a.dummy + lane_off;
  uint4 ring[P][NW][4];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const size_t o = (size_t)gi * tstride + (size_t)(kb0 + p) * BLOCK_ELEMS + lane_off;
    const bool in = p < nvb;
    const uint16_t* const b1 = in ? W + o : dummy;
    const uint16_t* const b2 = in ? W2 + o : dummy;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      ring[p][0][c] = load_stream(b1 + c * 512);
      if (NW == 2) ring[p][NW - 1][c] = load_stream(b2 + c * 512);
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
  float* const part = a.part + (size_t)s * a.part_split;
  float* const sink = a.sink + lane * 4;
  for (int j = 0; j < n_my; ++j) {
    const int tile = gi + j * G;
    // the ring's refills for the next tile; after the last tile they read the
    // small zero block instead (cache-resident, not another weight chunk)
    const bool more = j + 1 < n_my;
    const size_t t_base = (size_t)tile * tstride + (size_t)kb0 * BLOCK_ELEMS + lane_off;
    const size_t tn_base = t_base + (size_t)G * tstride;
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
        const size_t o = (next ? tn_base : t_base) + (size_t)qb * BLOCK_ELEMS;
        const uint16_t* const b1 = in ? W + o : dummy;
        const uint16_t* const b2 = in ? W2 + o : dummy;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          ring[r][0][c] = load_stream(b1 + c * 512);
          if (NW == 2) ring[r][NW - 1][c] = load_stream(b2 + c * 512);
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

}  // namespace

size_t gemm_dummy_elems() { return (size_t)BLOCK_ELEMS; }

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
  const int per = (p.n_tiles + G - 1) / G;
  p.G = (p.n_tiles + per - 1) / per;
  p.nw = nw;
  p.ldp = p.n_tiles * TILE_ROWS * nw;
  p.off2 = p.n_tiles * TILE_ROWS;
  return p;
}

size_t gemm_part_floats(int M, int N, int K, int nw, int target_wgs) {
  const GemmPlan p = plan_gemm(M, N, K, nw, target_wgs);
  return (size_t)p.S * M * p.ldp;
}

void launch_gemm(const uint16_t* X, int ldx, int M, const uint16_t* W, const uint16_t* W2, int N,
                 int K, float* part, float* sink, const uint16_t* dummy, const GemmScratch& sc,
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
  a.dummy = dummy;
  const dim3 grid(pl.S * pl.G);
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
