// bf16 MFMA contraction for gfx950: C[M,N] = alpha * sum_seg A_seg[M,K] B_seg[N,K]^T (+ C).
//
// Both operands are K-contiguous ("NT"): every contraction of the backward is brought to
// this layout by the kernels that produce its operands (transposed planes are written
// once, in the layout the contraction reads). Several (A, B) segments over the same K
// are summed in one pass: that is how fp32-valued operands enter as a sum of exact bf16
// terms. Products of bf16 values are exact in the fp32 accumulator.
//
// Tile 128 x 128 x 64, 256 threads (4 wave64s in 2 x 2, 64 x 64 per wave = 4 x 4 MFMA
// 16x16x32 tiles), double-buffered LDS with a 16-byte row pad (row stride 144 B keeps
// the 16 rows read by one ds_read_b128 on distinct banks). Workgroups are renumbered so
// that the tiles of one XCD are contiguous in row-major tile order (shared A panels in
// that XCD's L2).
#include "bsp_kernels.h"

namespace bsp {

constexpr int GBK = 64, GPAD = 72;

// Block tile BM x BN, 256 threads as a WGM x WGN grid of wave64s; each wave owns a
// (BM / WGM) x (BN / WGN) tile of 16 x 16 MFMA results.
template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmArgs g) {
  static_assert(WGM * WGN == 4, "four waves");
  constexpr int TM = BM / WGM, TN = BN / WGN, FM = TM / 16, FN = TN / 16;
  constexpr int LA = BM / 32, LB = BN / 32;  // 16-byte loads per thread per chunk
  __shared__ __attribute__((aligned(16))) u16 sA[2][BM][GPAD];
  __shared__ __attribute__((aligned(16))) u16 sB[2][BN][GPAD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int tiles_n = (g.N + BN - 1) / BN;
  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);  // XCD-contiguous tiles
  const int bm = (bid / tiles_n) * BM, bn = (bid % tiles_n) * BN;

  const int nch = (g.K + GBK - 1) / GBK;
  const int total = nch * g.nseg;

  const int lrow = tid >> 3, lk = (tid & 7) * 8;
  uint4 ra[LA], rb[LB];
  auto gload = [&](int c) {
    const int seg = c / nch;
    const int k0 = (c - seg * nch) * GBK + lk;
    const u16* A = g.A[seg];
    const u16* B = g.B[seg];
    const bool ka = k0 < g.K;
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      const int r = lrow + 32 * i;
      ra[i] = (bm + r < g.M && ka) ? *(const uint4*)(A + (int64_t)(bm + r) * g.lda + k0) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      const int r = lrow + 32 * i;
      rb[i] = (bn + r < g.N && ka) ? *(const uint4*)(B + (int64_t)(bn + r) * g.ldb + k0) : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LA; ++i) *(uint4*)&sA[buf][lrow + 32 * i][lk] = ra[i];
#pragma unroll
    for (int i = 0; i < LB; ++i) *(uint4*)&sB[buf][lrow + 32 * i][lk] = rb[i];
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (total > 0) {
    gload(0);
    sstore(0);
  }
  __syncthreads();
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  for (int c = 0; c < total; ++c) {
    const int buf = c & 1;
    if (c + 1 < total) gload(c + 1);
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 32) {
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[i] = *(const bf16x8*)&sA[buf][wm * TM + i * 16 + fr][kk + fk];
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[j] = *(const bf16x8*)&sB[buf][wn * TN + j * 16 + fr][kk + fk];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (c + 1 < total) sstore(buf ^ 1);
    __syncthreads();
  }

  // D[i][j] of a 16x16 tile sits in lane (j + 16 * (i / 4)), register i % 4.
  const int oc = lane & 15, orow = (lane >> 4) * 4;
  const float alpha = g.alpha_dev ? g.alpha * *g.alpha_dev : g.alpha;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = bn + wn * TN + j * 16 + oc;
      if (n >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = bm + wm * TM + i * 16 + orow + r;
        if (m < g.M) {
          float* p = g.C + (int64_t)m * g.ldc + n;
          const float v = alpha * acc[i][j][r];
          *p = g.accumulate ? *p + v : v;
        }
      }
    }
  }
}

template <int BM, int BN, int WGM, int WGN>
static bs_status launch_gemm_cfg(const GemmArgs& g, hipStream_t st) {
  const int64_t tiles = (int64_t)((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  if (tiles > 0x7FFFFFFF) return BS_ESHAPE;
  ProfScope prof("gemm", st);
  gemm_nt_kernel<BM, BN, WGM, WGN><<<(unsigned)tiles, 256, 0, st>>>(g);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_gemm(const GemmArgs& g, hipStream_t st) {
  if (g.M <= 0 || g.N <= 0) return BS_OK;
  if (g.nseg < 1 || g.nseg > GEMM_MAX_SEG) return BS_EINVAL;
  if ((g.K & 7) || (g.lda & 7) || (g.ldb & 7)) return BS_ESHAPE;
  if (g.K == 0) return g.accumulate ? BS_OK : launch_fill2d(g.C, g.M, g.N, g.ldc, 0.0f, st);
#ifdef BSP_GEMM_CFG
  return BSP_GEMM_CFG(g, st);
#else
  // 256 x 256 tiles once they still give every CU a tile; 128 x 128 below that
  const int64_t big = (int64_t)((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (big >= 256) return launch_gemm_cfg<256, 256, 2, 2>(g, st);
  return launch_gemm_cfg<128, 128, 2, 2>(g, st);
#endif
}

}  // namespace bsp
