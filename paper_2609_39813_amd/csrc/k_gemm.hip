// bf16 MFMA contraction for gfx950: C[M,N] = alpha * sum_seg A_seg[M,K] B_seg[N,K]^T (+ C).
//
// Both operands are K-contiguous ("NT"): every contraction of the backward is brought to
// this layout by the kernels that produce its operands (transposed planes are written
// once, in the layout the contraction reads). Several (A, B) segments over the same K
// are summed in one pass: that is how fp32-valued operands enter as a sum of exact bf16
// terms. Products of bf16 values are exact in the fp32 accumulator.
//
// Two kernels. The pipelined kernel (K a multiple of 64) moves operand tiles straight from
// global memory into LDS (buffer_load_dwordx4 ... lds, no register staging) in 64-deep
// chunks, so that every operand row of a chunk is one full 128-byte line; two LDS stages
// (128 KB for a 256 x 256 tile) hold the chunk being computed and the next one. A 256 x 256
// block tile is split over 8 wave64s of 128 x 64 (8 x 4 MFMA 16x16x32 tiles, accumulators in
// AGPRs): at 128 accumulator registers a wave fits twice per SIMD, so one wave's MFMAs run
// while the other waits on a load issue or the barrier. The 16-byte unit u of row r sits at unit u ^ (r & 7) of its LDS row, so the
// rows one ds_read_b128 serves together fall on distinct banks. The operand loads go through
// buffer resources that end with the tile's last valid row (rows past M or N read as zero).
// The instruction order of the main loop is fixed in source (scheduling barriers): LDS reads
// of the next k-step and the global loads of the chunk after next are spread between the
// MFMAs, one barrier per chunk. Shapes with fewer tiles than CUs split K over blocks into
// fp32 partials that one more kernel sums in a fixed order (the result does not depend on
// timing). The register-staged kernel below serves the other shapes.
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
  const float alpha = gemm_alpha(g);
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
// A stage holds a 64-deep K chunk: every operand row is one 128-byte line. The 16-byte unit u
// of row r sits at unit u ^ swz(r) of its LDS row, so that the rows one ds_read_b128 serves
// together fall on distinct banks.
constexpr int LBK = 64, LNST = 2;
__device__ __forceinline__ int swz_of(int r) { return r & 7; }
__device__ __forceinline__ int lds_swz(int r, int u) { return r * 128 + ((u ^ swz_of(r)) << 4); }

// Block tile BM x BN, WGM x WGN wave64s, each owning a (BM / WGM) x (BN / WGN) tile. F16: the
// operands hold fp16 values (v_mfma_f32_16x16x32_f16), else bf16.
template <int BM, int BN, int WGM, int WGN, bool F16>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_lds_kernel(GemmArgs g, int cps) {
  constexpr int NW = WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN, FM = WM / 16, FN = WN / 16;
  constexpr int AI = BM / (8 * NW), BI = BN / (8 * NW), LPC = AI + BI;  // 1-KB loads (8 rows) per wave per chunk
  static_assert(AI * 8 * NW == BM && BI * 8 * NW == BN, "loads cover the tile");
  constexpr int STAGE = (BM + BN) * 128;
  __shared__ __attribute__((aligned(1024))) char smem[LNST * STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN, ntile = tiles_m * tiles_n;
  const int nblk = gridDim.x;
  int bid = blockIdx.x;
  if ((nblk & 7) == 0) bid = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int zs = bid / ntile, tile = bid - zs * ntile;
  // a batched launch's member z (batched launches do not split K), else the split
  const int zb = g.batch > 1 ? zs : 0, split = g.batch > 1 ? 0 : zs;
  const int64_t oA = (int64_t)zb * g.sA, oB = (int64_t)zb * g.sB;
  // groups of GM tile rows: consecutive tiles (one XCD's share) form a GM-row patch, so the
  // A and B panels they read overlap in that XCD's L2
  constexpr int GM = 4;
  const int group = tile / (GM * tiles_n), in_group = tile - group * GM * tiles_n;
  const int first_m = group * GM, gsz = min(tiles_m - first_m, GM);
  const int bm = (first_m + in_group % gsz) * BM, bn = (in_group / gsz) * BN;
  const int nch = g.K / LBK, total = nch * g.nseg;
  const int c0 = split * cps;
  const int n = min(total, c0 + cps) - c0;

  // Operand tiles are read through buffer resources whose range ends with the tile's last
  // valid row: rows past M (N) read as zero (their products are never stored) and cost no
  // memory traffic. Load i of this wave fills rows (wave * AI + i) * 8 .. +7 of A (then B):
  // lane l writes row l / 8 at unit position l % 8, which holds logical unit (l % 8) ^ swz(row);
  // swz(row) = swz(l / 8) because the row's other terms are multiples of 8. One per-lane byte
  // offset per operand; the load index and the k position enter as scalar offsets.
  const int rows_a = min(g.M - bm, BM), rows_b = min(g.N - bn, BN);
  const uint32_t lane_a = (uint32_t)(((wave * AI * 8 + (lane >> 3)) * g.lda + (((lane & 7) ^ swz_of(lane >> 3)) << 3)) * 2);
  const uint32_t lane_b = (uint32_t)(((wave * BI * 8 + (lane >> 3)) * g.ldb + (((lane & 7) ^ swz_of(lane >> 3)) << 3)) * 2);
  const uint32_t step_a = (uint32_t)(8 * g.lda * 2), step_b = (uint32_t)(8 * g.ldb * 2);
  auto rsrc = [](const u16* base, int64_t row0, int rows, int64_t ld) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)(base + row0 * ld), (short)0, (int)(rows * ld * 2), 0x00020000);
  };
  // The next chunk to load: segment, k offset and the segment's resources (wave-uniform).
  // Past the last chunk of the contraction the position wraps to the start of the last
  // segment: the loop body is branch-free, and the surplus loads land in a stage that is
  // never read again.
  int iss_seg = c0 / nch, iss_k = (c0 - iss_seg * nch) * LBK;
  __amdgpu_buffer_rsrc_t ra = rsrc(g.A[iss_seg] + oA, bm, rows_a, g.lda);
  __amdgpu_buffer_rsrc_t rb = rsrc(g.B[iss_seg] + oB, bn, rows_b, g.ldb);
  auto issue_one = [&](int st, int i) {
    char* base = smem + st * STAGE;
    if (i < AI)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (void __attribute__((address_space(3)))*)(base + (wave * AI + i) * 1024),
                                               16, lane_a, (uint32_t)iss_k * 2 + i * step_a, 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rb, (void __attribute__((address_space(3)))*)(base + BM * 128 + (wave * BI + i - AI) * 1024), 16, lane_b,
          (uint32_t)iss_k * 2 + (i - AI) * step_b, 0, 0);
  };
  // Kept out of the MFMA regions: the rare segment switch is a branch with scalar loads.
  auto advance = [&]() {
    iss_k += LBK;
    if (iss_k == g.K) {
      iss_k = 0;
      if (++iss_seg < g.nseg) {
        ra = rsrc(g.A[iss_seg] + oA, bm, rows_a, g.lda);
        rb = rsrc(g.B[iss_seg] + oB, bn, rows_b, g.ldb);
      }
    }
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int fr = lane & 15, fc = lane >> 4;
  bf16x8 fa[2][FM], fb[2][FN];
  // MFMA t of a k-step, in row-major (i, j) order
  auto mfma_t = [&](int buf, int t) {
    const int i = t / FN, j = t % FN;
    if constexpr (F16)
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, fa[buf][i]),
                                                         __builtin_bit_cast(halfx8, fb[buf][j]), acc[i][j], 0, 0, 0);
    else
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[buf][i], fb[buf][j], acc[i][j], 0, 0, 0);
  };
  // read q of a k-step's fragments: B first (the first MFMAs use every B fragment), then A
  auto read_q = [&](int st, int s, int q, bf16x8* a, bf16x8* b) {
    const char* base = smem + st * STAGE;
    if (q < FN)
      b[q] = *(const bf16x8*)(base + BM * 128 + lds_swz(wn * WN + q * 16 + fr, fc + 4 * s));
    else
      a[q - FN] = *(const bf16x8*)(base + lds_swz(wm * WM + (q - FN) * 16 + fr, fc + 4 * s));
  };
  // wait until at most vm of this wave's loads are pending and its fragment reads are done,
  // then a barrier without a memory fence (a fence would drain the prefetch too)
#define BS_LAND(vm)                                                                             \
  do {                                                                                          \
    __builtin_amdgcn_s_waitcnt(((vm) & 15) | (((vm) >> 4) << 14) | (7 << 4)); /* lgkmcnt(0) */ \
    asm volatile("s_barrier" ::: "memory");                                                     \
  } while (0)
  static_assert(LPC < 64, "vmcnt range");

  // Prologue: chunks 0 and 1 in flight; chunk 0 landed; its first k-step in registers.
#pragma unroll
  for (int st = 0; st < 2; ++st) {
#pragma unroll
    for (int i = 0; i < LPC; ++i) issue_one(st, i);
    advance();
  }
  BS_LAND(LPC);
#pragma unroll
  for (int q = 0; q < FM + FN; ++q) read_q(0, 0, q, fa[0], fb[0]);

  // Chunk c (stage c & 1), two k-steps of 32; the fragments alternate between two register
  // sets (k-step 0 computes from set 0 and fills set 1, k-step 1 the reverse).
  // k-step 0: its MFMAs, with the fragments of k-step 1 (same stage, landed) read in between.
  // k-step 1: the MFMAs of the first PA fragment rows; then chunk c + 1 is awaited and every
  //   wave has finished reading chunk c; the loads of chunk c + 2 go into chunk c's stage and
  //   the first fragments of chunk c + 1 are read, both between the remaining MFMAs: one read
  //   per MFMA, one load per LSP MFMAs, evenly over all of them (a burst of loads stalls the
  //   wave at issue and with it its MFMAs).
  // The instruction order is fixed in source: a scheduling barrier closes every MFMA's group
  // (its load, its read), so reads are issued well before their use. The last iteration reads
  // a stage of surplus data that is never used.
  constexpr int NM = FM * FN;                  // MFMAs per k-step
  constexpr int RD = FM + FN;                  // fragment reads per k-step
  constexpr int PA = FM >= 4 ? FM / 4 : 1;     // rows before the barrier
  constexpr int NA = PA * FN, NB = NM - NA;    // MFMAs before / after the barrier
  constexpr int M0 = NM / RD >= 2 ? 2 : 1;     // k-step 0: one read per M0 MFMAs
  constexpr int LSP = NB / LPC > 0 ? NB / LPC : 1;  // k-step 1: one load per LSP MFMAs
  static_assert(RD <= NB && LPC <= NB, "k-step 1 holds the reads and loads");
  for (int c = 0; c < n; ++c) {
    const int st = c & 1;
#pragma unroll
    for (int q = 0; q < RD; ++q) {
      read_q(st, 1, q, fa[1], fb[1]);
#pragma unroll
      for (int t = q * M0; t < (q + 1) * M0; ++t) mfma_t(0, t);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int t = RD * M0; t < NM; ++t) mfma_t(0, t);
    __builtin_amdgcn_sched_barrier(0);

#pragma unroll
    for (int t = 0; t < NA; ++t) mfma_t(1, t);
    __builtin_amdgcn_sched_barrier(0);
    BS_LAND(0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int p = 0; p < NB; ++p) {
      if (p % LSP == 0 && p / LSP < LPC) issue_one(st, p / LSP);
      if (p < RD) read_q(st ^ 1, 0, p, fa[0], fb[0]);
      mfma_t(1, NA + p);
      __builtin_amdgcn_sched_barrier(0);
    }
    advance();
  }
  // no load into LDS may outlive the block (the CU hands its LDS to the next block)
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
#undef BS_LAND

  // D[i][j] of a 16x16 tile sits in lane (j + 16 * (i / 4)), register i % 4.
  const int oc = lane & 15, orow = (lane >> 4) * 4;
  float* out = g.part ? g.part + (int64_t)split * g.M * g.N : g.C + (int64_t)zb * g.sC;
  const int64_t ldo = g.part ? g.N : g.ldc;
  const float alpha = g.part ? 1.0f : gemm_alpha(g, zb);
  const bool acc_in = !g.part && g.accumulate;
  float mx = 0.0f;
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
          mx = fmaxf(mx, fabsf(v));
        }
      }
    }
  }
  if (g.amax && !g.part) wave_amax_to_slot(mx, g.amax);  // split partials: the split sum takes it
}

// C = alpha * sum_s part[s] (+ C), splits summed in order
__global__ __launch_bounds__(256) void gemm_split_sum_kernel(GemmArgs g, int splits) {
  const int64_t mn = (int64_t)g.M * g.N;
  const float alpha = gemm_alpha(g);
  float mx = 0.0f;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < mn; i += (int64_t)gridDim.x * blockDim.x) {
    float v = g.part[i];
    for (int s = 1; s < splits; ++s) v += g.part[(int64_t)s * mn + i];
    const int64_t m = i / g.N, nn = i - m * g.N;
    float* p = g.C + m * g.ldc + nn;
    *p = g.accumulate ? *p + alpha * v : alpha * v;
    mx = fmaxf(mx, fabsf(alpha * v));
  }
  if (g.amax) block_amax_to_slot(mx, g.amax);
}

template <int BM, int BN, int WGM, int WGN, bool F16>
static bs_status launch_gemm_lds(const GemmArgs& g0, hipStream_t st) {
  GemmArgs g = g0;
  const int64_t tiles = (int64_t)((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  const int total = (g.K / LBK) * g.nseg;
  // split K while the tiles leave CUs idle, keeping at least 16 chunks (1024 of K) per block. One
  // block fits a CU (its LDS), so blocks beyond the 256 CUs run in a second round: the split count
  // minimizes the makespan ceil(tiles * splits / 256) / splits (e.g. 48 tiles: 5 splits in one round
  // of 240 blocks, not 6 in two rounds of 288)
  int splits = 1;
  if (g.batch > 1) g.part = nullptr;  // batch members fill the CUs
  if (g.part && tiles < 256) {
    const int64_t by_k = total / 16;
    const int64_t by_ws = g.part_cap / ((int64_t)g.M * g.N);
    const int64_t top = std::max<int64_t>(1, std::min((256 + tiles - 1) / tiles, std::min(by_k, by_ws)));
    double best = 2.0;
    for (int64_t sp = 1; sp <= top; ++sp) {
      const double span = (double)((tiles * sp + 255) / 256) / (double)sp;
      if (span < best - 1e-12) {
        best = span;
        splits = (int)sp;
      }
    }
  }
  const int cps = (total + splits - 1) / splits;
  splits = (total + cps - 1) / cps;
  if (splits == 1) g.part = nullptr;
  const int64_t nblocks = tiles * (g.batch > 1 ? g.batch : splits);
  if (nblocks > 0x7FFFFFFF) return BS_ESHAPE;
  {
    ProfScope prof("gemm", st, gemm_flops(g), gemm_exec_flops(g));
    gemm_lds_kernel<BM, BN, WGM, WGN, F16><<<(unsigned)nblocks, 64 * WGM * WGN, 0, st>>>(g, cps);
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
  ProfScope prof("gemm", st, gemm_flops(g), gemm_exec_flops(g));
  gemm_nt_kernel<BM, BN, WGM, WGN><<<(unsigned)tiles, 256, 0, st>>>(g);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_gemm(const GemmArgs& g, hipStream_t st) {
  if (g.M <= 0 || g.N <= 0) return BS_OK;
  if (g.nseg < 1 || g.nseg > GEMM_MAX_SEG) return BS_EINVAL;
  if ((g.K & 7) || (g.lda & 7) || (g.ldb & 7) || g.lda < g.K || g.ldb < g.K) return BS_ESHAPE;
  if (g.amax && g.accumulate) return BS_EINVAL;
  if (g.batch < 1 || (g.batch > 1 && (g.sA < 0 || g.sB < 0 || g.sC < 0 || g.s_alpha2 < 0))) return BS_EINVAL;
  if (g.K == 0) return g.accumulate ? BS_OK : launch_fill2d(g.C, g.M, g.N, g.ldc, 0.0f, st);
  // pipelined kernel for 64-aligned K and 16-byte aligned operands
  // (buffer offsets of one 256-row tile fit in 31 bits)
  bool lds_ok = (g.K % LBK) == 0 && g.M >= 1 && g.N >= 1 && g.lda < (1 << 21) && g.ldb < (1 << 21);
  for (int i = 0; i < g.nseg; ++i) lds_ok = lds_ok && ((uintptr_t)g.A[i] & 15) == 0 && ((uintptr_t)g.B[i] & 15) == 0;
  const bool big_tiles = (int64_t)g.M * g.N >= (int64_t)256 * 256 * 16;
  if (lds_ok && g.f16)
    return big_tiles ? launch_gemm_lds<256, 256, 2, 4, true>(g, st) : launch_gemm_lds<128, 128, 2, 2, true>(g, st);
  if (g.f16 || g.amax || g.batch > 1) return BS_EINVAL;  // fp16 operands, maxima, batches: the pipelined kernel only
  if (lds_ok)
    return big_tiles ? launch_gemm_lds<256, 256, 2, 4, false>(g, st) : launch_gemm_lds<128, 128, 2, 2, false>(g, st);
  // 256 x 256 tiles once they still give every CU a tile; 128 x 128 below that
  const int64_t big = (int64_t)((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (big >= 256) return launch_gemm_cfg<256, 256, 2, 2>(g, st);
  return launch_gemm_cfg<128, 128, 2, 2>(g, st);
}

}  // namespace bsp
