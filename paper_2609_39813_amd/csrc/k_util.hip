// Utility kernels: fills, bf16 operand planes (copy / split / transpose), and the trial
// statistics reducer.
#include "bsp_kernels.h"

namespace bsp {

__global__ void init_diag_only(bs_diag* diag) {
  if (threadIdx.x == 0) {
    diag->nonfinite = 0;
    diag->n_saturated = 0;
    diag->amax = 0.0f;
    diag->scale = 1.0f;
  }
}

bs_status launch_init_diag(bs_diag* diag, hipStream_t st) {
  init_diag_only<<<1, 64, 0, st>>>(diag);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

__global__ void fill2d_kernel(float* p, int64_t rows, int64_t cols, int64_t ld, float v) {
  const int64_t n = rows * cols;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[(i / cols) * ld + (i % cols)] = v;
}
__global__ void fill_f64_kernel(double* p, int64_t n, double v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

bs_status launch_fill2d(float* p, int64_t rows, int64_t cols, int64_t ld, float v, hipStream_t st) {
  const int64_t n = rows * cols;
  if (n <= 0) return BS_OK;
  const int64_t want = (n + 255) / 256;
  fill2d_kernel<<<(unsigned)(want < 4096 ? want : 4096), 256, 0, st>>>(p, rows, cols, ld, v);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_fill_f64(double* p, int64_t n, double v, hipStream_t st) {
  if (n <= 0) return BS_OK;
  const int64_t want = (n + 255) / 256;
  fill_f64_kernel<<<(unsigned)(want < 4096 ? want : 4096), 256, 0, st>>>(p, n, v);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// ------------------------------------------------------------------------------------
// bf16 planes of a [R, C] matrix: value * scale split into nterms bf16 terms.
// ------------------------------------------------------------------------------------
struct PlaneOut {
  u16* p[3];
};

__device__ __forceinline__ void split_to(float v, int nterms, u16 (&o)[3]) {
  if (nterms == 1) {
    o[0] = bf16_bits(v);
    o[1] = o[2] = 0;
  } else {
    split3(v, o[0], o[1], o[2]);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void planes_rows_kernel(const T* __restrict__ in, int64_t R, int64_t C, int64_t ldi,
                                                          PlaneOut out, int nterms, int64_t ldo, float scale) {
  const int64_t n = R * ldo;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / ldo, c = i - r * ldo;
    const float v = c < C ? load_f32(in, r * ldi + c) * scale : 0.0f;
    u16 o[3];
    split_to(v, nterms, o);
    for (int p = 0; p < nterms; ++p) out.p[p][i] = o[p];
  }
}

// The same planes of an fp32 matrix 4 elements per thread (C, ldi and ldo multiples of 4, 16-byte
// aligned input rows, 8-byte aligned planes): one index division per 4 elements, 16-byte loads,
// 8-byte stores per plane.
__global__ __launch_bounds__(256) void planes_rows4_kernel(const float* __restrict__ in, int64_t R, int64_t C,
                                                           int64_t ldi, PlaneOut out, int nterms, int64_t ldo,
                                                           float scale) {
  const int64_t q = ldo / 4, n = R * q;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / q, c = 4 * (i - r * q);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c < C) v = *(const float4*)(in + r * ldi + c);
    const float x[4] = {v.x * scale, v.y * scale, v.z * scale, v.w * scale};
    u16 o[4][3];
#pragma unroll
    for (int k = 0; k < 4; ++k) split_to(x[k], nterms, o[k]);
#pragma unroll
    for (int p = 0; p < 3; ++p)
      if (p < nterms)
        *(uint2*)(out.p[p] + 4 * i) = make_uint2((uint32_t)o[0][p] | ((uint32_t)o[1][p] << 16),
                                                 (uint32_t)o[2][p] | ((uint32_t)o[3][p] << 16));
  }
}

// Transposed: out_p[c * ldo + r] for r < ldo (zero for r >= R). Tile 64 x 64 through LDS.
template <typename T>
__global__ __launch_bounds__(256) void planes_t_kernel(const T* __restrict__ in, int64_t R, int64_t C, int64_t ldi,
                                                       PlaneOut out, int nterms, int64_t ldo, float scale) {
  __shared__ u16 tile[3][64][66];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int rr = ty + 4 * i;
    const int64_t r = r0 + rr, c = c0 + tx;
    const float v = (r < R && c < C) ? load_f32(in, r * ldi + c) * scale : 0.0f;
    u16 o[3];
    split_to(v, nterms, o);
    for (int p = 0; p < nterms; ++p) tile[p][rr][tx] = o[p];
  }
  __syncthreads();
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int cc = ty + 4 * i;
    const int64_t c = c0 + cc, r = r0 + tx;
    if (c < C && r < ldo)
      for (int p = 0; p < nterms; ++p) out.p[p][c * ldo + r] = tile[p][tx][cc];
  }
}

// The transpose of a bf16 [R, C] matrix (C and ldi multiples of 8, 16-byte aligned rows) into
// [C][ldo] with zeros in rows R .. ldo - 1 of every output row: one 64 x 64 tile per block,
// 16-byte loads and stores, the tile held in LDS with rows padded to 144 bytes.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const u16* __restrict__ in, int64_t R, int64_t C,
                                                             int64_t ldi, u16* __restrict__ out, int64_t ldo) {
  __shared__ __attribute__((aligned(16))) u16 tile[64][72];
  const int t = threadIdx.x, q = (t & 7) * 8;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int rr = (t >> 3) + 32 * pass;
    const int64_t r = r0 + rr, c = c0 + q;
    const uint4 v = (r < R && c < C) ? *(const uint4*)(in + r * ldi + c) : make_uint4(0, 0, 0, 0);
    *(uint4*)&tile[rr][q] = v;
  }
  __syncthreads();
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int cc = (t >> 3) + 32 * pass;
    const int64_t c = c0 + cc;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (uint32_t)tile[q + 2 * i][cc] | ((uint32_t)tile[q + 2 * i + 1][cc] << 16);
    if (c < C) *(uint4*)(out + c * ldo + r0 + q) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// The transposed planes of an fp32 [R, C] matrix (C and ldi multiples of 4, 16-byte aligned rows,
// ldo a multiple of 64) split into nterms bf16 terms per value (the split of planes_t_kernel): a
// 64 x 64 tile goes into LDS as fp32 (rows padded to 65 words, so both the row writes and the
// column reads below fall on distinct banks); a thread then splits 8 consecutive rows of one
// column and stores them as one 16-byte piece per plane, eight threads covering 128 bytes of an
// output row.
__global__ __launch_bounds__(256) void transpose_split_f32_kernel(const float* __restrict__ in, int64_t R, int64_t C,
                                                                  int64_t ldi, PlaneOut out, int nterms, int64_t ldo,
                                                                  float scale) {
  __shared__ float tile[64][65];
  const int c4 = threadIdx.x & 15, rq = threadIdx.x >> 4;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rr = rq + 16 * i;
    const int64_t r = r0 + rr, c = c0 + 4 * c4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < R && c < C) v = *(const float4*)(in + r * ldi + c);
    tile[rr][4 * c4 + 0] = v.x * scale;
    tile[rr][4 * c4 + 1] = v.y * scale;
    tile[rr][4 * c4 + 2] = v.z * scale;
    tile[rr][4 * c4 + 3] = v.w * scale;
  }
  __syncthreads();
  const int rg = threadIdx.x & 7;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int cc = (threadIdx.x >> 3) + 32 * pass;
    const int64_t c = c0 + cc;
    if (c >= C) continue;
    u16 o[8][3];
#pragma unroll
    for (int i = 0; i < 8; ++i) split_to(tile[8 * rg + i][cc], nterms, o[i]);
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      if (p >= nterms) break;
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (uint32_t)o[2 * i][p] | ((uint32_t)o[2 * i + 1][p] << 16);
      *(uint4*)(out.p[p] + c * ldo + r0 + 8 * rg) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// The row-major planes of an fp32 matrix, 8 elements per thread (C and ldi multiples of 4, ldo a
// multiple of 8, 16-byte aligned input rows and planes): grid x over 2048-column pieces of a row,
// grid y over rows; two 16-byte loads, one 16-byte store per plane, no index division.
__global__ __launch_bounds__(256) void planes_rows8_kernel(const float* __restrict__ in, int64_t R, int64_t C,
                                                           int64_t ldi, PlaneOut out, int nterms, int64_t ldo,
                                                           float scale) {
  const int64_t c = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (c >= ldo) return;
  for (int64_t r = blockIdx.y; r < R; r += gridDim.y) {
    float4 v0 = make_float4(0.f, 0.f, 0.f, 0.f), v1 = v0;
    if (c < C) v0 = *(const float4*)(in + r * ldi + c);
    if (c + 4 < C) v1 = *(const float4*)(in + r * ldi + c + 4);
    const float x[8] = {v0.x * scale, v0.y * scale, v0.z * scale, v0.w * scale,
                        v1.x * scale, v1.y * scale, v1.z * scale, v1.w * scale};
    u16 o[8][3];
#pragma unroll
    for (int k = 0; k < 8; ++k) split_to(x[k], nterms, o[k]);
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      if (p >= nterms) break;
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (uint32_t)o[2 * i][p] | ((uint32_t)o[2 * i + 1][p] << 16);
      *(uint4*)(out.p[p] + r * ldo + c) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

bs_status launch_planes(const void* in, bs_dtype dt, int64_t R, int64_t C, int64_t ldi, bool transpose,
                        u16* const* outp, int nterms, int64_t ldo, float scale, hipStream_t st) {
  if (nterms < 1 || nterms > 3) return BS_EINVAL;
  PlaneOut out{{outp[0], nterms > 1 ? outp[1] : nullptr, nterms > 2 ? outp[2] : nullptr}};
  if (transpose) {
    if (C <= 0 || ldo <= 0) return BS_OK;
    dim3 grid((unsigned)((C + 63) / 64), (unsigned)((ldo + 63) / 64));
    const bool vec = dt == BS_BF16 && nterms == 1 && scale == 1.0f && C % 8 == 0 && ldi % 8 == 0 && ldo % 64 == 0 &&
                     ((uintptr_t)in & 15) == 0 && ((uintptr_t)outp[0] & 15) == 0;
    bool vecf = dt == BS_F32 && C % 4 == 0 && ldi % 4 == 0 && ldo % 64 == 0 && ((uintptr_t)in & 15) == 0;
    for (int p = 0; p < nterms; ++p) vecf = vecf && ((uintptr_t)outp[p] & 15) == 0;
    if (vec)
      transpose_bf16_kernel<<<grid, 256, 0, st>>>((const u16*)in, R, C, ldi, outp[0], ldo);
    else if (vecf)
      transpose_split_f32_kernel<<<grid, 256, 0, st>>>((const float*)in, R, C, ldi, out, nterms, ldo, scale);
    else if (dt == BS_F32)
      planes_t_kernel<float><<<grid, 256, 0, st>>>((const float*)in, R, C, ldi, out, nterms, ldo, scale);
    else
      planes_t_kernel<u16><<<grid, 256, 0, st>>>((const u16*)in, R, C, ldi, out, nterms, ldo, scale);
  } else {
    const int64_t n = R * ldo;
    if (n <= 0) return BS_OK;
    const int64_t want = (n + 255) / 256;
    const unsigned blocks = (unsigned)(want < 8192 ? want : 8192);
    bool vec8 = dt == BS_F32 && C % 4 == 0 && ldi % 4 == 0 && ldo % 8 == 0 && ((uintptr_t)in & 15) == 0;
    for (int p = 0; p < nterms; ++p) vec8 = vec8 && ((uintptr_t)outp[p] & 15) == 0;
    bool vec4 = dt == BS_F32 && C % 4 == 0 && ldi % 4 == 0 && ldo % 4 == 0 && ((uintptr_t)in & 15) == 0;
    for (int p = 0; p < nterms; ++p) vec4 = vec4 && ((uintptr_t)outp[p] & 7) == 0;
    if (vec8) {
      const dim3 grid((unsigned)((ldo / 8 + 255) / 256), (unsigned)(R < 65535 ? R : 65535));
      planes_rows8_kernel<<<grid, 256, 0, st>>>((const float*)in, R, C, ldi, out, nterms, ldo, scale);
    } else if (vec4) {
      const int64_t want4 = (n / 4 + 255) / 256;
      planes_rows4_kernel<<<(unsigned)(want4 < 8192 ? want4 : 8192), 256, 0, st>>>((const float*)in, R, C, ldi, out,
                                                                                   nterms, ldo, scale);
    } else if (dt == BS_F32)
      planes_rows_kernel<float><<<blocks, 256, 0, st>>>((const float*)in, R, C, ldi, out, nterms, ldo, scale);
    else
      planes_rows_kernel<u16><<<blocks, 256, 0, st>>>((const u16*)in, R, C, ldi, out, nterms, ldo, scale);
  }
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// ------------------------------------------------------------------------------------
// The operands of a move's contractions as scaled two-term fp16 splits, from one read of the move
// (and of the gradient it moves): its transposed planes (the weight use), those of gradient +
// move, and its row-major planes (the move's own propagation). A 64 x 64 tile per block, staged
// through LDS as in the transposed split above.
// ------------------------------------------------------------------------------------
__device__ __forceinline__ const float* move_at(const MoveSrc& m, int64_t t, int64_t c) {
  if (m.rows) return m.rows + t * m.ldi + c;
  // 32-bit division (the launcher bounds rows and columns below 2^31)
  const uint32_t which = (uint32_t)c / (uint32_t)m.d, cc = (uint32_t)c - which * (uint32_t)m.d;  // Q, K or V; column
  const uint32_t b = (uint32_t)t / (uint32_t)m.S, s = (uint32_t)t - b * (uint32_t)m.S;
  return m.heads[which] + ((((int64_t)b * m.H + (cc >> 6)) * m.S + s) << 6) + (cc & 63);
}

// BASE: the planes of base + move too (a second LDS tile)
template <bool BASE>
__global__ __launch_bounds__(256) void split_move_f16_kernel(MoveSrc src, const float* __restrict__ base, int64_t ldb,
                                                             int64_t R, int64_t C, F16Scale sc, PlaneOut tM,
                                                             PlaneOut tS, int64_t ldo, PlaneOut rows, int64_t ldr) {
  __shared__ float tile[64][65];
  __shared__ float tileS[BASE ? 64 : 1][65];
  const float a = amax_of_slots(sc.amax_a), b = sc.amax_b ? amax_of_slots(sc.amax_b) : 0.0f;
  const int e = f16_scale_exp(fmaxf(a, b)) - (sc.amax_b ? 1 : 0);
  const float scl = ldexpf(1.0f, e);
  if (sc.inv_out && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *sc.inv_out = ldexpf(1.0f, -e);
  const int c4 = threadIdx.x & 15, rq = threadIdx.x >> 4;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rr = rq + 16 * i;
    const int64_t r = r0 + rr, c = c0 + 4 * c4;
    const bool in = r < R && c < C;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f), w = v;
    if (in) {
      v = *(const float4*)move_at(src, r, c);
      if (BASE) {
        const float4 g = *(const float4*)(base + r * ldb + c);
        w = make_float4(g.x + v.x, g.y + v.y, g.z + v.z, g.w + v.w);
      }
    }
    const float x[4] = {v.x * scl, v.y * scl, v.z * scl, v.w * scl};
#pragma unroll
    for (int q = 0; q < 4; ++q) tile[rr][4 * c4 + q] = x[q];
    if (BASE) {
      tileS[rr][4 * c4 + 0] = w.x * scl;
      tileS[rr][4 * c4 + 1] = w.y * scl;
      tileS[rr][4 * c4 + 2] = w.z * scl;
      tileS[rr][4 * c4 + 3] = w.w * scl;
    }
    if (rows.p[0] && in) {
      u16 hi[4], lo[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) split2_f16(x[q], hi[q], lo[q]);
      *(uint2*)(rows.p[0] + r * ldr + c) = make_uint2((uint32_t)hi[0] | ((uint32_t)hi[1] << 16),
                                                      (uint32_t)hi[2] | ((uint32_t)hi[3] << 16));
      *(uint2*)(rows.p[1] + r * ldr + c) = make_uint2((uint32_t)lo[0] | ((uint32_t)lo[1] << 16),
                                                      (uint32_t)lo[2] | ((uint32_t)lo[3] << 16));
    }
  }
  __syncthreads();
  // a thread splits 8 consecutive rows of one column: one 16-byte piece per plane
  const int rg = threadIdx.x & 7;
  auto put = [&](float (*t)[65], const PlaneOut& out, int cc, int64_t c) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      u16 h0, l0, h1, l1;
      split2_f16(t[8 * rg + 2 * i][cc], h0, l0);
      split2_f16(t[8 * rg + 2 * i + 1][cc], h1, l1);
      h[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
      l[i] = (uint32_t)l0 | ((uint32_t)l1 << 16);
    }
    *(uint4*)(out.p[0] + c * ldo + r0 + 8 * rg) = make_uint4(h[0], h[1], h[2], h[3]);
    *(uint4*)(out.p[1] + c * ldo + r0 + 8 * rg) = make_uint4(l[0], l[1], l[2], l[3]);
  };
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int cc = (threadIdx.x >> 3) + 32 * pass;
    const int64_t c = c0 + cc;
    if (c >= C) continue;
    put(tile, tM, cc, c);
    if (BASE) put(tileS, tS, cc, c);
  }
}

bs_status launch_split_move(const MoveSrc& m, const float* base, int64_t ldb, int64_t R, int64_t C, F16Scale sc,
                            u16* const* tM, u16* const* tS, int64_t ldo, u16* const* rows, int64_t ldr,
                            hipStream_t st) {
  auto a16 = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  if (!sc.amax_a || !tM || !tM[0] || !tM[1] || (base && (!tS || !tS[0] || !tS[1])) ||
      (rows && (!rows[0] || !rows[1])))
    return BS_EINVAL;
  if (R < 0) return BS_EINVAL;
  if (C <= 0 || ldo <= 0) return BS_OK;  // R = 0: the transposed planes are zero
  bool ok = C % 4 == 0 && ldo % 64 == 0 && ldo >= R && a16(tM[0]) && a16(tM[1]);
  if (m.rows) {
    ok = ok && m.ldi % 4 == 0 && m.ldi >= C && a16(m.rows);
  } else {
    // head-major: 64-wide heads, C / d of Q, K, V, R = B S rows
    ok = ok && m.d > 0 && m.d % 64 == 0 && m.H * 64 == m.d && m.S > 0 && R % m.S == 0 && C % m.d == 0 &&
         C / m.d <= 3 && R < ((int64_t)1 << 31) && C < ((int64_t)1 << 31);
    for (int64_t i = 0; ok && i < C / m.d; ++i) ok = m.heads[i] && a16(m.heads[i]);
  }
  if (base) ok = ok && ldb % 4 == 0 && ldb >= C && a16(base) && a16(tS[0]) && a16(tS[1]);
  if (rows) ok = ok && ldr % 4 == 0 && ldr >= C && ((uintptr_t)rows[0] & 7) == 0 && ((uintptr_t)rows[1] & 7) == 0;
  if (!ok) return BS_EINVAL;
  const PlaneOut pm{{tM[0], tM[1], nullptr}};
  const PlaneOut ps{{base ? tS[0] : nullptr, base ? tS[1] : nullptr, nullptr}};
  const PlaneOut pr{{rows ? rows[0] : nullptr, rows ? rows[1] : nullptr, nullptr}};
  const dim3 grid((unsigned)((C + 63) / 64), (unsigned)(ldo / 64));
  if (base)
    split_move_f16_kernel<true><<<grid, 256, 0, st>>>(m, base, ldb, R, C, sc, pm, ps, ldo, pr, ldr);
  else
    split_move_f16_kernel<false><<<grid, 256, 0, st>>>(m, base, ldb, R, C, sc, pm, ps, ldo, pr, ldr);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// fp16 of a bf16 tensor scaled by 2^e (the max in slots), 2^-e to inv_out
__global__ __launch_bounds__(256) void scale_f16_kernel(const u16* __restrict__ in, int64_t n,
                                                        const uint32_t* __restrict__ slots, u16* __restrict__ out,
                                                        float* __restrict__ inv_out) {
  const int e = f16_scale_exp(amax_of_slots(slots));
  const float scl = ldexpf(1.0f, e);
  if (inv_out && blockIdx.x == 0 && threadIdx.x == 0) *inv_out = ldexpf(1.0f, -e);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    out[i] = f16_bits(__uint_as_float((uint32_t)in[i] << 16) * scl);
}

bs_status launch_scale_f16(const u16* in, int64_t n, const uint32_t* slots, u16* out, float* inv_out, hipStream_t st) {
  if (n < 0 || (n > 0 && (!in || !slots || !out))) return BS_EINVAL;
  if (n == 0) return BS_OK;
  const int64_t want = (n + 255) / 256;
  scale_f16_kernel<<<(unsigned)(want < 4096 ? want : 4096), 256, 0, st>>>(in, n, slots, out, inv_out);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// ------------------------------------------------------------------------------------
// Trial statistics: per column j of delta [K][m], mean over trials (fp64, trials in
// order), sample variance by a second pass, se = sd / sqrt(K); block partial sums of
// mean^2, ref^2 and se^2 (fp64), combined in block order by one more kernel.
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void trial_stats_kernel(const float* __restrict__ delta, int K, int64_t m,
                                                          const float* __restrict__ g_ref, float* __restrict__ mean_err,
                                                          float* __restrict__ se, double* __restrict__ part) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  double mean = 0.0, var = 0.0, ref = 0.0;
  if (j < m) {
    // mean = d_1 + (1/K) sum_k (d_k - d_1): exactly d_1 when every trial agrees
    const double d1 = delta[j];
    double s = 0.0;
    for (int k = 1; k < K; ++k) s += (double)delta[(int64_t)k * m + j] - d1;
    mean = d1 + s / K;
    double q = 0.0;
    for (int k = 0; k < K; ++k) {
      const double e = (double)delta[(int64_t)k * m + j] - mean;
      q += e * e;
    }
    var = K > 1 ? q / (K - 1) / K : 0.0;
    mean_err[j] = (float)mean;
    if (se) se[j] = (float)sqrt(var);
    if (g_ref) ref = g_ref[j];
  }
  __shared__ double red[3][4];
  double v[3] = {mean * mean, ref * ref, var};
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int i = 0; i < 3; ++i) {
    const double s = wave_sum_f64(v[i]);
    if (lane == 0) red[i][w] = s;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int i = threadIdx.x;
    part[(int64_t)blockIdx.x * 3 + i] = ((red[i][0] + red[i][1]) + red[i][2]) + red[i][3];
  }
}

// One block of 256 threads: thread i adds the partials of blocks i, i + 256, ... in order, then a
// fixed pairwise tree (offsets 128, 64, ..., 1) combines the threads (deterministic).
__global__ __launch_bounds__(256) void trial_summary_kernel(const double* __restrict__ part, int64_t nblk,
                                                            double* __restrict__ summary) {
  __shared__ double red[3][256];
  double s[3] = {0.0, 0.0, 0.0};
  for (int64_t b = threadIdx.x; b < nblk; b += 256)
    for (int i = 0; i < 3; ++i) s[i] += part[b * 3 + i];
  for (int i = 0; i < 3; ++i) red[i][threadIdx.x] = s[i];
  __syncthreads();
  for (int off = 128; off >= 1; off >>= 1) {
    if ((int)threadIdx.x < off)
      for (int i = 0; i < 3; ++i) red[i][threadIdx.x] += red[i][threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    summary[0] = sqrt(red[0][0]);
    summary[1] = sqrt(red[1][0]);
    summary[2] = red[2][0] > 0.0 ? red[0][0] / red[2][0] : __builtin_nan("");
  }
}

bs_status launch_policy_bias(const float* delta, int K, int64_t m, const float* g_ref, float* mean_err, float* se,
                             double* summary, double* ws, hipStream_t st) {
  const int64_t nblk = (m + 255) / 256;
  if (nblk > 0)
    trial_stats_kernel<<<(unsigned)nblk, 256, 0, st>>>(delta, K, m, g_ref, mean_err, se, ws);
  if (summary) trial_summary_kernel<<<1, 256, 0, st>>>(ws, nblk, summary);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
