// Thin-M bf16 GEMM on gfx950 MFMA: Y[m][n] = sum_k X[m][k] * W[n][k].
//
// The decode path multiplies a few dozen activation rows (tree nodes) by
// large weight matrices, so the kernel is bound by streaming W from HBM once.
// Layout of the work:
//  - one workgroup of 8 waves owns 16*NT consecutive rows of W (and of W2 for
//    the SwiGLU pair) and all M rows of X (MT tiles of 16); the 8 waves split
//    K into contiguous ranges of 128-element blocks, and their partial tiles
//    are summed through LDS in wave order, so no workgroup ever waits for
//    another and the result does not depend on timing;
//  - v_mfma_f32_16x16x32_bf16 with A = W rows and B = X^T columns.  The K
//    index inside one MFMA may be any permutation shared by A and B, so a
//    lane loads 32 physically contiguous bf16 of its W row (the four lanes of
//    a row cover 256 contiguous bytes per block) and the same 32 columns of
//    its X row;
//  - the loads of the next P-1 blocks are in flight while a block's MFMAs
//    run (a ring of P register stages), which keeps enough bytes outstanding
//    per CU to cover HBM latency;
//  - the weight may be given as up to three row segments (e.g. the q, k and v
//    projections) that behave as one matrix of the summed height.
#include "msd_internal.h"

namespace msd {

namespace {

constexpr int KB = 128;     // K elements per block
constexpr int WAVES = 8;

template <int MT, int NT, int NW>
struct Frag {
  uint4 w[NW][NT][4];
  uint4 x[MT][4];
};

// Block load.  Rows past N or M were clamped to row 0 by the caller (they
// only feed output rows that are never stored).  Full blocks (GUARD false)
// load without any per-lane condition, which is what lets the compiler keep
// several blocks in flight; the single partial block at the end of K
// (K % 128 != 0) uses GUARD and zeroes the W columns past K.
template <int MT, int NT, int NW, bool GUARD>
MSD_DEV void load_block(Frag<MT, NT, NW>& f, const uint16_t* const (&wrow)[NW][NT],
                        const uint16_t* const (&xrow)[MT], int k, int K) {
  // k is this lane's first column of the block; K % 8 == 0
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int kk = k + 8 * c;
    const bool ok = !GUARD || kk < K;
    const int kc = ok ? kk : K - 8;
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int s = 0; s < NT; ++s) {
        const uint4 v = *reinterpret_cast<const uint4*>(wrow[w][s] + kc);
        f.w[w][s][c] = ok ? v : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
    for (int t = 0; t < MT; ++t) f.x[t][c] = *reinterpret_cast<const uint4*>(xrow[t] + kc);
  }
}

template <int MT, int NT, int NW>
MSD_DEV void mma_block(f32x4 (&acc)[NW][NT][MT], const Frag<MT, NT, NW>& f) {
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int s = 0; s < NT; ++s)
#pragma unroll
        for (int t = 0; t < MT; ++t)
          acc[w][s][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              as_bf16x8(f.w[w][s][c]), as_bf16x8(f.x[t][c]), acc[w][s][t], 0, 0, 0);
}

template <int MT, int NT, int EPI, int P>
__global__ __launch_bounds__(512) void k_gemm(GemmArgs a) {
  constexpr int NW = (EPI == EPI_SILU) ? 2 : 1;
  constexpr int TILE = NW * NT * MT * 4;  // floats per lane per wave
  __shared__ float red[WAVES / 2][TILE][64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16 * NT;

  const uint16_t* wrow[NW][NT];
#pragma unroll
  for (int s = 0; s < NT; ++s) {
    const int n = n0 + 16 * s + i;
    const int nn = n < a.N ? n : 0;
    // 16-row tiles never straddle a segment (segment heights are multiples of 16)
    const int seg = (nn < a.seg_end[0]) ? 0 : (nn < a.seg_end[1] ? 1 : 2);
    const int base = seg == 0 ? 0 : a.seg_end[seg - 1];
    wrow[0][s] = a.Wseg[seg] + (size_t)(nn - base) * a.K;
    if (NW == 2) wrow[NW - 1][s] = a.W2 + (size_t)nn * a.K;
  }
  const uint16_t* xrow[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int m = t * 16 + i;
    xrow[t] = a.X + (size_t)(m < a.M ? m : 0) * a.ldx;
  }

  f32x4 acc[NW][NT][MT];
#pragma unroll
  for (int w = 0; w < NW; ++w)
#pragma unroll
    for (int s = 0; s < NT; ++s)
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[w][s][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // contiguous, balanced range of full blocks for this wave; the trip count
  // is uniform across the wave and the prefetch index is clamped rather than
  // guarded
  const int nkb = a.K / KB;
  const int kb0 = (nkb * wave) / WAVES;
  const int kb1 = (nkb * (wave + 1)) / WAVES;
  if (kb0 < kb1) {
    const int last = kb1 - 1;
    Frag<MT, NT, NW> ring[P];
#pragma unroll
    for (int p = 0; p < P; ++p)
      load_block<MT, NT, NW, false>(ring[p], wrow, xrow, min(kb0 + p, last) * KB + 32 * g, a.K);
    int kb = kb0;
    for (; kb + P <= kb1; kb += P) {
#pragma unroll
      for (int p = 0; p < P; ++p) {
        mma_block<MT, NT, NW>(acc, ring[p]);
        load_block<MT, NT, NW, false>(ring[p], wrow, xrow, min(kb + p + P, last) * KB + 32 * g,
                                      a.K);
      }
    }
#pragma unroll
    for (int p = 0; p < P; ++p)
      if (p < kb1 - kb) mma_block<MT, NT, NW>(acc, ring[p]);
  }
  if (wave == WAVES - 1 && nkb * KB < a.K) {
    Frag<MT, NT, NW> f;
    load_block<MT, NT, NW, true>(f, wrow, xrow, nkb * KB + 32 * g, a.K);
    mma_block<MT, NT, NW>(acc, f);
  }

  // pairwise reduction over the 8 waves through LDS:
  // ((w0 + w4) + (w2 + w6)) + ((w1 + w5) + (w3 + w7))
#pragma unroll
  for (int half = 4; half >= 1; half >>= 1) {
    if (wave >= half && wave < 2 * half) {
#pragma unroll
      for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int s = 0; s < NT; ++s)
#pragma unroll
          for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              red[wave - half][((w * NT + s) * MT + t) * 4 + r][lane] = acc[w][s][t][r];
    }
    __syncthreads();
    if (wave < half) {
#pragma unroll
      for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int s = 0; s < NT; ++s)
#pragma unroll
          for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              acc[w][s][t][r] += red[wave][((w * NT + s) * MT + t) * 4 + r][lane];
    }
    __syncthreads();
  }
  if (wave != 0) return;

  // C layout of the 16x16 MFMA: lane holds column (lane & 15) = output row
  // m, register r holds W row 4*(lane/16) + r of the 16-row tile.
#pragma unroll
  for (int s = 0; s < NT; ++s)
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = t * 16 + i;
        const int n = n0 + 16 * s + 4 * g + r;
        if (m >= a.M || n >= a.N) continue;
        const float v0 = acc[0][s][t][r];
        const size_t o = (size_t)m * a.ldo + n;
        if (EPI == EPI_F32) {
          a.out_f32[o] = v0;
        } else if (EPI == EPI_RESID) {
          a.out_f32[o] += v0;
        } else if (EPI == EPI_BF16) {
          a.out_bf16[o] = f2bf(v0);
        } else {
          const float v1 = acc[NW - 1][s][t][r];
          a.out_bf16[o] = f2bf(v0 / (1.f + __expf(-v0)) * v1);
        }
      }
}

// ring depth: three stages when a stage is at most 64 VGPRs, else two
template <int MT, int NT, int NW>
constexpr int ring_depth() { return (16 * NT * NW + 16 * MT) <= 64 ? 3 : 2; }

template <int MT, int NT>
void dispatch_epi(int epi, dim3 grid, const GemmArgs& a, hipStream_t st) {
  constexpr int P1 = ring_depth<MT, NT, 1>();
  constexpr int P2 = ring_depth<MT, NT, 2>();
  switch (epi) {
    case EPI_F32: hipLaunchKernelGGL((k_gemm<MT, NT, EPI_F32, P1>), grid, dim3(512), 0, st, a); break;
    case EPI_BF16: hipLaunchKernelGGL((k_gemm<MT, NT, EPI_BF16, P1>), grid, dim3(512), 0, st, a); break;
    case EPI_RESID: hipLaunchKernelGGL((k_gemm<MT, NT, EPI_RESID, P1>), grid, dim3(512), 0, st, a); break;
    default: hipLaunchKernelGGL((k_gemm<MT, NT, EPI_SILU, P2>), grid, dim3(512), 0, st, a); break;
  }
}

}  // namespace

void launch_gemm(int epi, const uint16_t* X, int ldx, int M, const uint16_t* const* Wseg,
                 const int* seg_rows, int n_seg, const uint16_t* W2, int K, float* out_f32,
                 uint16_t* out_bf16, int ldo, const GemmScratch& s, hipStream_t st) {
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
  // wider row tiles for wide matrices (fewer re-reads of X) as long as the
  // grid still covers every CU
  const int tiles16 = (N + 15) / 16;
  int nt = 1;
  if (tiles16 >= 2 * s.target_wgs) nt = 2;
  if (M > 32) nt = 1;
  for (int m0 = 0; m0 < M; m0 += 64) {
    const int mc = (M - m0) < 64 ? (M - m0) : 64;
    GemmArgs a = base;
    a.X = X + (size_t)m0 * ldx;
    a.ldx = ldx;
    a.M = mc;
    a.W2 = W2;
    a.N = N;
    a.K = K;
    a.out_f32 = out_f32 ? out_f32 + (size_t)m0 * ldo : nullptr;
    a.out_bf16 = out_bf16 ? out_bf16 + (size_t)m0 * ldo : nullptr;
    a.ldo = ldo;
    dim3 grid((N + 16 * nt - 1) / (16 * nt));
    if (mc <= 16) {
      if (nt == 2) dispatch_epi<1, 2>(epi, grid, a, st); else dispatch_epi<1, 1>(epi, grid, a, st);
    } else if (mc <= 32) {
      if (nt == 2) dispatch_epi<2, 2>(epi, grid, a, st); else dispatch_epi<2, 1>(epi, grid, a, st);
    } else {
      dispatch_epi<4, 1>(epi, grid, a, st);
    }
  }
}

void launch_gemm(int epi, const uint16_t* X, int ldx, int M, const uint16_t* W,
                 const uint16_t* W2, int N, int K, float* out_f32, uint16_t* out_bf16,
                 int ldo, const GemmScratch& s, hipStream_t st) {
  launch_gemm(epi, X, ldx, M, &W, &N, 1, W2, K, out_f32, out_bf16, ldo, s, st);
}

}  // namespace msd
