// bf16 MFMA contraction for gfx950: C[M,N] = alpha * sum_seg A_seg[M,K] B_seg[N,K]^T (+ C).
//
// Both operands are K-contiguous ("NT"): every contraction of the backward is brought to
// this layout by the kernels that produce its operands (transposed planes are written
// once, in the layout the contraction reads). Several (A, B) segments over the same K
// are summed in one pass: that is how fp32-valued operands enter as a sum of exact bf16
// terms. Products of bf16 values are exact in the fp32 accumulator.
//
// Two kernels. The pipelined kernel (K a multiple of 32) moves operand tiles straight from
// global memory into LDS (global_load_lds_dwordx4, no register staging) through a ring of
// four 32-deep stages, three chunks ahead of the MFMAs; a 256 x 256 block tile is split over
// 4 wave64s of 128 x 128 (8 x 8 MFMA 16x16x32 tiles, accumulators in AGPRs). Rows of a stage
// are 64 B; the 16-byte chunk c of row r sits at chunk c ^ ((r >> 1) & 3), so the eight rows
// a ds_read_b128 phase touches fall on distinct banks. Shapes with fewer tiles than CUs split
// K over blocks into fp32 partials that one more kernel sums in a fixed order (the result
// does not depend on timing). The register-staged kernel below serves the other shapes.
//
// Register-staged kernel: tile 128 x 128 x 64 or 256 x 256 x 64, 256 threads (4 wave64s in
// 2 x 2), double-buffered LDS with a 16-byte row pad (row stride 144 B keeps the 16 rows read
// by one ds_read_b128 on distinct banks).
//
// Both renumber workgroups so that the tiles of one XCD are contiguous in row-major tile order
// (shared A panels in that XCD's L2).
#include <algorithm>

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

// ------------------------------------------------------------------------------------
// pipelined kernel
// ------------------------------------------------------------------------------------
#ifndef BSP_GEMM_STAGES
#define BSP_GEMM_STAGES 4
#endif
constexpr int LBK = 32, LNST = BSP_GEMM_STAGES;

__device__ __forceinline__ int lds_swz(int r, int c) { return r * 64 + ((c ^ ((r >> 1) & 3)) << 4); }

// s_waitcnt with vmcnt = n and the other counters left at their maxima (gfx9 encoding)
#define BS_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (15 << 8))

template <int BM, int BN>
__global__ __launch_bounds__(256) void gemm_lds_kernel(GemmArgs g, int cps) {
  constexpr int WM = BM / 2, WN = BN / 2, FM = WM / 16, FN = WN / 16;
  constexpr int AI = BM / 64, BI = BN / 64, LPC = AI + BI;  // 1-KB loads per wave per stage
  constexpr int STAGE = (BM + BN) * 64;
  __shared__ __attribute__((aligned(1024))) char smem[LNST * STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN, ntile = tiles_m * tiles_n;
  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int split = bid / ntile, tile = bid - split * ntile;
  // groups of GM tile rows: consecutive tiles (one XCD's share) form a GM-row patch, so the
  // A and B panels they read overlap in that XCD's L2
  constexpr int GM = 4;
  const int group = tile / (GM * tiles_n), in_group = tile - group * GM * tiles_n;
  const int first_m = group * GM, gsz = min(tiles_m - first_m, GM);
  const int bm = (first_m + in_group % gsz) * BM, bn = (in_group / gsz) * BN;
  const int nch = g.K / LBK, total = nch * g.nseg;
  const int c0 = split * cps;
  const int n = min(total, c0 + cps) - c0;

  // Load i of this wave fills rows (wave * AI + i) * 16 .. +15 of A (then B): lane l writes
  // row l / 4, chunk position l % 4, which holds logical chunk (l % 4) ^ ((row >> 1) & 3).
  // Rows past M (N) repeat the last row; their products are never stored.
  int64_t offa[AI], offb[BI];
#pragma unroll
  for (int i = 0; i < AI; ++i) {
    const int r = (wave * AI + i) * 16 + (lane >> 2);
    offa[i] = (int64_t)min(bm + r, g.M - 1) * g.lda + (((lane & 3) ^ ((r >> 1) & 3)) << 3);
  }
#pragma unroll
  for (int i = 0; i < BI; ++i) {
    const int r = (wave * BI + i) * 16 + (lane >> 2);
    offb[i] = (int64_t)min(bn + r, g.N - 1) * g.ldb + (((lane & 3) ^ ((r >> 1) & 3)) << 3);
  }
  // the next chunk to load: segment, k offset and the segment's operands (wave-uniform)
  int iss_seg = c0 / nch, iss_k = (c0 - iss_seg * nch) * LBK;
  const u16* pa = g.A[iss_seg];
  const u16* pb = g.B[iss_seg];
  auto issue = [&](int st) {
    char* base = smem + st * STAGE;
#pragma unroll
    for (int i = 0; i < AI; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(pa + offa[i] + iss_k),
                                       (void __attribute__((address_space(3)))*)(base + (wave * AI + i) * 1024),
                                       16, 0, 0);
#pragma unroll
    for (int i = 0; i < BI; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(pb + offb[i] + iss_k),
                                       (void __attribute__((address_space(3)))*)(base + BM * 64 + (wave * BI + i) * 1024),
                                       16, 0, 0);
    iss_k += LBK;
    if (iss_k == g.K) {
      iss_k = 0;
      if (++iss_seg < g.nseg) {
        pa = g.A[iss_seg];
        pb = g.B[iss_seg];
      }
    }
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Software pipeline: the fragments of chunk c + 1 are read from LDS while the MFMAs of
  // chunk c run; chunk c + 3 is in flight from global memory.
  const int fr = lane & 15, fc = lane >> 4;
  bf16x8 fa[2][FM], fb[2][FN];
  auto read_frags = [&](int c, bf16x8* a, bf16x8* b) {
    const char* base = smem + (c % LNST) * STAGE;
#pragma unroll
    for (int i = 0; i < FM; ++i) a[i] = *(const bf16x8*)(base + lds_swz(wm * WM + i * 16 + fr, fc));
#pragma unroll
    for (int j = 0; j < FN; ++j) b[j] = *(const bf16x8*)(base + BM * 64 + lds_swz(wn * WN + j * 16 + fr, fc));
  };
  auto mfmas = [&](const bf16x8* a, const bf16x8* b) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  };
  // wait until chunk c has landed (at most the loads of the chunks issued after it pending),
  // then a barrier without a memory fence (the fence would drain the prefetches too)
  auto wait_chunks = [&](int after) {  // at most `after` chunks' loads still pending
    static_assert(LNST >= 3 && LNST <= 5, "waits below cover up to three chunks in flight");
    if (LNST >= 5 && after >= 3)
      BS_WAIT_VM(3 * LPC);
    else if (LNST >= 4 && after >= 2)
      BS_WAIT_VM(2 * LPC);
    else if (after >= 1)
      BS_WAIT_VM(LPC);
    else
      BS_WAIT_VM(0);
  };
  auto land = [&](int x) {
    // chunks issued when x is awaited: up to min(n - 1, x + LNST - 3)
    wait_chunks(min(n - 1, x + LNST - 3) - x);
    asm volatile("s_barrier" ::: "memory");
  };

#pragma unroll
  for (int st = 0; st < LNST - 1; ++st)
    if (st < n) issue(st);
  wait_chunks(min(n - 1, LNST - 2));  // chunk 0 with chunks 1 .. LNST - 2 still in flight
  asm volatile("s_barrier" ::: "memory");
  read_frags(0, fa[0], fb[0]);

  for (int c = 0; c + 1 < n; ++c) {
    land(c + 1);
    if (c + LNST - 1 < n) issue((c + LNST - 1) % LNST);
    read_frags(c + 1, fa[1], fb[1]);
    mfmas(fa[0], fb[0]);
    // interleave: one fragment read after every few MFMAs
#pragma unroll
    for (int q = 0; q < FM + FN; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, (FM * FN) / (FM + FN), 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[0][i] = fa[1][i];
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[0][j] = fb[1][j];
  }
  mfmas(fa[0], fb[0]);

  // D[i][j] of a 16x16 tile sits in lane (j + 16 * (i / 4)), register i % 4.
  const int oc = lane & 15, orow = (lane >> 4) * 4;
  float* out = g.part ? g.part + (int64_t)split * g.M * g.N : g.C;
  const int64_t ldo = g.part ? g.N : g.ldc;
  const float alpha = g.part ? 1.0f : (g.alpha_dev ? g.alpha * *g.alpha_dev : g.alpha);
  const bool acc_in = !g.part && g.accumulate;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int nn = bn + wn * WN + j * 16 + oc;
      if (nn >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = bm + wm * WM + i * 16 + orow + r;
        if (m < g.M) {
          float* p = out + (int64_t)m * ldo + nn;
          const float v = alpha * acc[i][j][r];
          *p = acc_in ? *p + v : v;
        }
      }
    }
  }
}

// C = alpha * sum_s part[s] (+ C), splits summed in order
__global__ __launch_bounds__(256) void gemm_split_sum_kernel(GemmArgs g, int splits) {
  const int64_t mn = (int64_t)g.M * g.N;
  const float alpha = g.alpha_dev ? g.alpha * *g.alpha_dev : g.alpha;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < mn; i += (int64_t)gridDim.x * blockDim.x) {
    float v = g.part[i];
    for (int s = 1; s < splits; ++s) v += g.part[(int64_t)s * mn + i];
    const int64_t m = i / g.N, nn = i - m * g.N;
    float* p = g.C + m * g.ldc + nn;
    *p = g.accumulate ? *p + alpha * v : alpha * v;
  }
}

template <int BM, int BN>
static bs_status launch_gemm_lds(const GemmArgs& g0, hipStream_t st) {
  GemmArgs g = g0;
  const int64_t tiles = (int64_t)((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  const int total = (g.K / LBK) * g.nseg;
  // split K while the tiles leave CUs idle, keeping at least 32 chunks (1024 of K) per block
  int splits = 1;
  if (g.part && tiles < 256) {
    const int64_t want = (256 + tiles - 1) / tiles;
    const int64_t by_k = total / 32;
    const int64_t by_ws = g.part_cap / ((int64_t)g.M * g.N);
    splits = (int)std::max<int64_t>(1, std::min(want, std::min(by_k, by_ws)));
  }
  const int cps = (total + splits - 1) / splits;
  splits = (total + cps - 1) / cps;
  if (splits == 1) g.part = nullptr;
  if (tiles * splits > 0x7FFFFFFF) return BS_ESHAPE;
  {
    ProfScope prof("gemm", st);
    gemm_lds_kernel<BM, BN><<<(unsigned)(tiles * splits), 256, 0, st>>>(g, cps);
    BS_CHECK_LAUNCH();
  }
  if (splits > 1) {
    const int64_t mn = (int64_t)g.M * g.N;
    const unsigned blocks = (unsigned)std::min<int64_t>((mn + 255) / 256, 8192);
    ProfScope prof("gemm_split_sum", st);
    gemm_split_sum_kernel<<<blocks, 256, 0, st>>>(g, splits);
    BS_CHECK_LAUNCH();
  }
  return BS_OK;
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
  if ((g.K & 7) || (g.lda & 7) || (g.ldb & 7) || g.lda < g.K || g.ldb < g.K) return BS_ESHAPE;
  if (g.K == 0) return g.accumulate ? BS_OK : launch_fill2d(g.C, g.M, g.N, g.ldc, 0.0f, st);
#ifdef BSP_GEMM_CFG
  return BSP_GEMM_CFG(g, st);
#else
  // pipelined kernel for 32-aligned K and 16-byte aligned operands
  bool lds_ok = (g.K % LBK) == 0 && g.M >= 1 && g.N >= 1;
  for (int i = 0; i < g.nseg; ++i) lds_ok = lds_ok && ((uintptr_t)g.A[i] & 15) == 0 && ((uintptr_t)g.B[i] & 15) == 0;
  if (lds_ok) {
    if ((int64_t)g.M * g.N >= (int64_t)256 * 256 * 16) return launch_gemm_lds<256, 256>(g, st);
    return launch_gemm_lds<128, 128>(g, st);
  }
  // 256 x 256 tiles once they still give every CU a tile; 128 x 128 below that
  const int64_t big = (int64_t)((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (big >= 256) return launch_gemm_cfg<256, 256, 2, 2>(g, st);
  return launch_gemm_cfg<128, 128, 2, 2>(g, st);
#endif
}

}  // namespace bsp
