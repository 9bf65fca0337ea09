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

constexpr int GBM = 128, GBN = 128, GBK = 64, GPAD = 72;

__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) u16 sA[2][GBM][GPAD];
  __shared__ __attribute__((aligned(16))) u16 sB[2][GBN][GPAD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_n = (g.N + GBN - 1) / GBN;
  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);  // XCD-contiguous tiles
  const int bm = (bid / tiles_n) * GBM, bn = (bid % tiles_n) * GBN;

  const int nch = (g.K + GBK - 1) / GBK;
  const int total = nch * g.nseg;

  // global -> register staging: 4 x 16 B of A and of B per thread
  const int lrow = tid >> 3, lk = (tid & 7) * 8;
  uint4 ra[4], rb[4];
  auto gload = [&](int c) {
    const int seg = c / nch;
    const int k0 = (c - seg * nch) * GBK + lk;
    const u16* A = g.A[seg];
    const u16* B = g.B[seg];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = lrow + 32 * i;
      const bool ka = k0 < g.K;
      ra[i] = (bm + r < g.M && ka) ? *(const uint4*)(A + (int64_t)(bm + r) * g.lda + k0) : make_uint4(0, 0, 0, 0);
      rb[i] = (bn + r < g.N && ka) ? *(const uint4*)(B + (int64_t)(bn + r) * g.ldb + k0) : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *(uint4*)&sA[buf][lrow + 32 * i][lk] = ra[i];
      *(uint4*)&sB[buf][lrow + 32 * i][lk] = rb[i];
    }
  };

  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

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
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *(const bf16x8*)&sA[buf][wm * 64 + i * 16 + fr][kk + fk];
#pragma unroll
      for (int j = 0; j < 4; ++j) bfr[j] = *(const bf16x8*)&sB[buf][wn * 64 + j * 16 + fr][kk + fk];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (c + 1 < total) sstore(buf ^ 1);
    __syncthreads();
  }

  // D[i][j] of a 16x16 tile sits in lane (j + 16 * (i / 4)), register i % 4.
  const int oc = lane & 15, orow = (lane >> 4) * 4;
  const float alpha = g.alpha_dev ? g.alpha * *g.alpha_dev : g.alpha;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = bn + wn * 64 + j * 16 + oc;
      if (n >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = bm + wm * 64 + i * 16 + orow + r;
        if (m < g.M) {
          float* p = g.C + (int64_t)m * g.ldc + n;
          const float v = alpha * acc[i][j][r];
          *p = g.accumulate ? *p + v : v;
        }
      }
    }
  }
}

bs_status launch_gemm(const GemmArgs& g, hipStream_t st) {
  if (g.M <= 0 || g.N <= 0) return BS_OK;
  if (g.nseg < 1 || g.nseg > GEMM_MAX_SEG) return BS_EINVAL;
  if ((g.K & 7) || (g.lda & 7) || (g.ldb & 7)) return BS_ESHAPE;
  const int64_t tiles = (int64_t)((g.M + GBM - 1) / GBM) * ((g.N + GBN - 1) / GBN);
  if (tiles > 0x7FFFFFFF) return BS_ESHAPE;
  if (g.K == 0) return g.accumulate ? BS_OK : launch_fill2d(g.C, g.M, g.N, g.ldc, 0.0f, st);
  ProfScope prof("gemm", st);
  gemm_nt_kernel<<<(unsigned)tiles, 256, 0, st>>>(g);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
