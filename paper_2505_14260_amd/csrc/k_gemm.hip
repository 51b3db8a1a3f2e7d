// Thin-M bf16 GEMM on gfx950 MFMA: Y[m][n] = sum_k X[m][k] * W[n][k].
//
// The decode path multiplies a few dozen activation rows (tree nodes) by
// large weight matrices, so the kernel is bound by streaming W from HBM once.
// Layout of the work:
//  - a workgroup is 4 waves; wave w owns 32 rows of W (n0 = 128*tile + 32*w)
//    and all M rows of X (MT tiles of 32), over a range of K blocks of 64;
//  - v_mfma_f32_32x32x16_bf16 with A = W rows, B = X^T columns.  The K
//    index inside one MFMA may be any permutation shared by A and B, so each
//    lane loads 32 physically contiguous bf16 of its W row (lanes l and l+32
//    cover one 128-byte line of a row) and the same 32 columns of its X row;
//  - split-K across workgroups with a deterministic reduction: partial tiles
//    go to scratch, the last workgroup of a tile (integer atomic counter)
//    sums them in split order and runs the epilogue, then resets the counter.
#include "msd_internal.h"

namespace msd {

namespace {

constexpr int KB = 64;  // K elements per block

template <int MT, int NW>
struct Frag {
  uint4 w[NW][4];
  uint4 x[MT][4];
};

template <int MT, int NW>
MSD_DEV void load_block(Frag<MT, NW>& f, const uint16_t* const* wrow, bool nvalid,
                        const uint16_t* const* xrow, const bool* mvalid, int k, int K) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int kk = k + 8 * c;
    const bool ok = kk < K;
#pragma unroll
    for (int w = 0; w < NW; ++w)
      f.w[w][c] = (ok && nvalid) ? *reinterpret_cast<const uint4*>(wrow[w] + kk)
                                 : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int t = 0; t < MT; ++t)
      f.x[t][c] = (ok && mvalid[t]) ? *reinterpret_cast<const uint4*>(xrow[t] + kk)
                                    : make_uint4(0, 0, 0, 0);
  }
}

template <int MT, int NW>
MSD_DEV void mma_block(f32x16 (&acc)[NW][MT], const Frag<MT, NW>& f) {
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int t = 0; t < MT; ++t)
        acc[w][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(f.w[w][c]),
                                                            as_bf16x8(f.x[t][c]),
                                                            acc[w][t], 0, 0, 0);
}

template <int MT, int EPI>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  constexpr int NW = (EPI == EPI_SILU) ? 2 : 1;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int tile = blockIdx.x / a.splits;
  const int split = blockIdx.x - tile * a.splits;
  const int i = lane & 31, h = lane >> 5;
  const int n0 = tile * 128 + wave * 32;
  const int kb0 = split * a.kb_per_split;
  const int kb1 = min(kb0 + a.kb_per_split, a.n_kblocks);

  const int nrow = n0 + i;
  const bool nvalid = nrow < a.N;
  const uint16_t* wrow[NW];
  wrow[0] = a.W + (size_t)(nvalid ? nrow : 0) * a.K;
  if (NW == 2) wrow[NW - 1] = a.W2 + (size_t)(nvalid ? nrow : 0) * a.K;
  const uint16_t* xrow[MT];
  bool mvalid[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int m = t * 32 + i;
    mvalid[t] = m < a.M;
    xrow[t] = a.X + (size_t)(mvalid[t] ? m : 0) * a.ldx;
  }

  f32x16 acc[NW][MT];
#pragma unroll
  for (int w = 0; w < NW; ++w)
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[w][t][r] = 0.f;

  if (kb0 < kb1) {
    Frag<MT, NW> cur;
    load_block<MT, NW>(cur, wrow, nvalid, xrow, mvalid, kb0 * KB + 32 * h, a.K);
    for (int kb = kb0; kb < kb1; ++kb) {
      Frag<MT, NW> nxt;
      if (kb + 1 < kb1)
        load_block<MT, NW>(nxt, wrow, nvalid, xrow, mvalid, (kb + 1) * KB + 32 * h, a.K);
      mma_block<MT, NW>(acc, cur);
      cur = nxt;
    }
  }

  if (a.splits > 1) {
    constexpr int TILE_FLOATS = NW * MT * 16 * 64;
    float* mine = a.partial + ((size_t)blockIdx.x * 4 + wave) * TILE_FLOATS;
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          __hip_atomic_store(mine + ((w * MT + t) * 16 + r) * 64 + lane, acc[w][t][r],
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __threadfence();
    __syncthreads();
    __shared__ int s_last;
    if (threadIdx.x == 0) {
      const int prev = atomicAdd(a.counters + tile, 1);
      s_last = (prev == a.splits - 1);
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    const float* base = a.partial + ((size_t)tile * a.splits * 4 + wave) * TILE_FLOATS;
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float s = 0.f;
          const int off = ((w * MT + t) * 16 + r) * 64 + lane;
          for (int sp = 0; sp < a.splits; ++sp) {
            const float v = (sp == split)
                                ? acc[w][t][r]
                                : __hip_atomic_load(base + (size_t)sp * 4 * TILE_FLOATS + off,
                                                    __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s += v;
          }
          acc[w][t][r] = s;
        }
    if (threadIdx.x == 0) a.counters[tile] = 0;
  }

  // C layout of the 32x32 MFMA: lane holds column (lane & 31) = output row m,
  // register r holds W row n0 + 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int m = t * 32 + i;
    if (m >= a.M) continue;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int n = n0 + 8 * (r >> 2) + 4 * h + (r & 3);
      if (n >= a.N) continue;
      const size_t o = (size_t)m * a.ldo + n;
      if (EPI == EPI_F32) {
        a.out_f32[o] = acc[0][t][r];
      } else if (EPI == EPI_RESID) {
        a.out_f32[o] += acc[0][t][r];
      } else if (EPI == EPI_BF16) {
        a.out_bf16[o] = f2bf(acc[0][t][r]);
      } else {
        const float g = acc[0][t][r], u = acc[NW - 1][t][r];
        a.out_bf16[o] = f2bf(g / (1.f + __expf(-g)) * u);
      }
    }
  }
}

template <int MT>
void dispatch_epi(int epi, dim3 grid, const GemmArgs& a, hipStream_t st) {
  switch (epi) {
    case EPI_F32: hipLaunchKernelGGL((k_gemm<MT, EPI_F32>), grid, dim3(256), 0, st, a); break;
    case EPI_BF16: hipLaunchKernelGGL((k_gemm<MT, EPI_BF16>), grid, dim3(256), 0, st, a); break;
    case EPI_RESID: hipLaunchKernelGGL((k_gemm<MT, EPI_RESID>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((k_gemm<MT, EPI_SILU>), grid, dim3(256), 0, st, a); break;
  }
}

}  // namespace

size_t gemm_partial_floats(int max_m, int max_n, int target_wgs) {
  (void)max_n;
  // splits * tiles <= max(target_wgs, tiles) and each split-K workgroup
  // stores 4 waves * NW(<=2) * MT(<=2) * 16 * 64 floats.
  (void)max_m;
  const size_t per_wg = 4 * 2 * 2 * 16 * 64;
  return per_wg * (size_t)(target_wgs * 2 + 64);
}

void launch_gemm(int epi, const uint16_t* X, int ldx, int M, const uint16_t* W,
                 const uint16_t* W2, int N, int K, float* out_f32, uint16_t* out_bf16,
                 int ldo, const GemmScratch& s, hipStream_t st) {
  const int n_tiles = (N + 127) / 128;
  const int n_kblocks = (K + KB - 1) / KB;
  const int mt_cap = 2;
  for (int m0 = 0; m0 < M; m0 += 32 * mt_cap) {
    const int mc = (M - m0) < 32 * mt_cap ? (M - m0) : 32 * mt_cap;
    const int MT = mc <= 32 ? 1 : 2;
    int splits = 1;
    if (n_tiles < s.target_wgs) {
      splits = (s.target_wgs + n_tiles - 1) / n_tiles;
      if (splits > n_kblocks) splits = n_kblocks;
      if (splits > 64) splits = 64;
    }
    int kb_per = (n_kblocks + splits - 1) / splits;
    splits = (n_kblocks + kb_per - 1) / kb_per;
    const int NW = (epi == EPI_SILU) ? 2 : 1;
    if (splits > 1) {
      const size_t need = (size_t)n_tiles * splits * 4 * NW * MT * 16 * 64;
      if (need > s.partial_floats || n_tiles > s.n_counters) {
        splits = 1;
        kb_per = n_kblocks;
      }
    }
    GemmArgs a;
    a.X = X + (size_t)m0 * ldx;
    a.ldx = ldx;
    a.M = mc;
    a.W = W;
    a.W2 = W2;
    a.N = N;
    a.K = K;
    a.splits = splits;
    a.kb_per_split = kb_per;
    a.n_kblocks = n_kblocks;
    a.partial = s.partial;
    a.counters = s.counters;
    a.out_f32 = out_f32 ? out_f32 + (size_t)m0 * ldo : nullptr;
    a.out_bf16 = out_bf16 ? out_bf16 + (size_t)m0 * ldo : nullptr;
    a.ldo = ldo;
    dim3 grid(n_tiles * splits);
    if (MT == 1)
      dispatch_epi<1>(epi, grid, a, st);
    else
      dispatch_epi<2>(epi, grid, a, st);
  }
}

}  // namespace msd
