// Elementwise kernels of the decoder layer: head / token permutations, SwiGLU forward and
// backward, residual adds, bf16 concatenation, and batched fixed-order sums of squares.
#include "k_layer.h"

namespace bsp {

static unsigned blocks_for(int64_t n, int64_t cap = 16384) {
  const int64_t want = (n + 255) / 256;
  return (unsigned)(want < 1 ? 1 : (want < cap ? want : cap));
}
#define GRID_LOOP(i, n) \
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < (n); i += (int64_t)gridDim.x * blockDim.x)

// QKV [T][3d] fp32 -> Q, K, V [B,H,S,dh] bf16 (round to nearest even)
__global__ void qkv_heads_kernel(const float* __restrict__ qkv, int B, int S, int H, int dh, u16* __restrict__ Q,
                                 u16* __restrict__ K, u16* __restrict__ V) {
  const int d = H * dh;
  const int64_t n = (int64_t)B * S * 3 * d;
  GRID_LOOP(i, n) {
    const int64_t t = i / (3 * d);
    const int col = (int)(i - t * 3 * d);
    const int which = col / d, hc = col - which * d, h = hc / dh, c = hc - h * dh;
    const int b = (int)(t / S), s = (int)(t - (int64_t)b * S);
    const int64_t o = (((int64_t)b * H + h) * S + s) * dh + c;
    (which == 0 ? Q : (which == 1 ? K : V))[o] = bf16_bits(qkv[i]);
  }
}

// The same, one block per token row, four consecutive columns per thread (dh % 4 == 0: the four
// stay in one head): a 16-byte load and an 8-byte store, 32-bit index arithmetic.
__global__ __launch_bounds__(256) void qkv_heads4_kernel(const float4* __restrict__ qkv, int S, int H, int dh,
                                                         u16* __restrict__ Q, u16* __restrict__ K,
                                                         u16* __restrict__ V) {
  const int d = H * dh, t = blockIdx.x, b = t / S, s = t - b * S;
  for (int c4 = threadIdx.x; c4 < 3 * d / 4; c4 += 256) {
    const int col = 4 * c4, which = col / d, hc = col - which * d, h = hc / dh, c = hc - h * dh;
    const float4 v = qkv[(int64_t)t * (3 * d / 4) + c4];
    const int64_t o = (((int64_t)b * H + h) * S + s) * dh + c;
    u16* const out = which == 0 ? Q : (which == 1 ? K : V);
    *(uint2*)(out + o) = make_uint2((uint32_t)bf16_bits(v.x) | ((uint32_t)bf16_bits(v.y) << 16),
                                    (uint32_t)bf16_bits(v.z) | ((uint32_t)bf16_bits(v.w) << 16));
  }
}

// [B,H,S,dh] <-> [T][H*dh] (row t = b*S + s); element size 4 (fp32) or 1 (codes)
template <typename E>
__global__ void heads_tokens_kernel(const E* __restrict__ in, E* __restrict__ out, int B, int S, int H, int dh,
                                    int to_tokens) {
  const int64_t n = (int64_t)B * H * S * dh;
  GRID_LOOP(i, n) {
    const int c = (int)(i % dh);
    const int64_t r = i / dh;
    const int s = (int)(r % S);
    const int64_t bh = r / S;
    const int h = (int)(bh % H), b = (int)(bh / H);
    const int64_t tok = ((int64_t)b * S + s) * (H * dh) + h * dh + c;
    if (to_tokens)
      out[tok] = in[i];
    else
      out[i] = in[tok];
  }
}

// The same permutations four elements at a time (dh a multiple of 4): one block per token row
// t = b S + s, whose d (or 3 d) values are 16-byte pieces of H head rows; 32-bit index math.
// heads -> tokens (to_tokens) or back, for 4-byte elements (E4 = float4) or 1-byte codes
// (E4 = uint32_t)
template <typename E4>
__global__ __launch_bounds__(256) void heads_tokens4_kernel(const E4* __restrict__ in, E4* __restrict__ out, int S,
                                                            int H, int dh, int to_tokens) {
  const int t = blockIdx.x, b = t / S, s = t - b * S;
  const int q = dh / 4, n = H * q;  // 4-element pieces per token row and per head row
  for (int k = threadIdx.x; k < n; k += blockDim.x) {
    const int h = k / q, c = k - h * q;
    const int64_t hm = (((int64_t)b * H + h) * S + s) * q + c, tk = (int64_t)t * n + k;
    if (to_tokens)
      out[tk] = in[hm];
    else
      out[hm] = in[tk];
  }
}
// dQ, dK, dV [B,H,S,dh] -> dQKV [T][3d], four elements at a time
__global__ __launch_bounds__(256) void dqkv_tokens4_kernel(const float4* __restrict__ dQ, const float4* __restrict__ dK,
                                                           const float4* __restrict__ dV, float4* __restrict__ out,
                                                           int S, int H, int dh) {
  const int t = blockIdx.x, b = t / S, s = t - b * S;
  const int q = dh / 4, n = H * q;
  for (int k = threadIdx.x; k < 3 * n; k += blockDim.x) {
    const int which = k / n, kk = k - which * n, h = kk / q, c = kk - h * q;
    const int64_t hm = (((int64_t)b * H + h) * S + s) * q + c;
    out[(int64_t)t * 3 * n + k] = (which == 0 ? dQ : (which == 1 ? dK : dV))[hm];
  }
}

// dQ, dK, dV [B,H,S,dh] -> dQKV [T][3d]
__global__ void dqkv_tokens_kernel(const float* __restrict__ dQ, const float* __restrict__ dK,
                                   const float* __restrict__ dV, float* __restrict__ out, int B, int S, int H, int dh) {
  const int d = H * dh;
  const int64_t n = (int64_t)B * S * 3 * d;
  GRID_LOOP(i, n) {
    const int64_t t = i / (3 * d);
    const int col = (int)(i - t * 3 * d);
    const int which = col / d, hc = col - which * d, h = hc / dh, c = hc - h * dh;
    const int b = (int)(t / S), s = (int)(t - (int64_t)b * S);
    const int64_t o = (((int64_t)b * H + h) * S + s) * dh + c;
    out[i] = (which == 0 ? dQ : (which == 1 ? dK : dV))[o];
  }
}

__global__ void bf16_to_f32_kernel(const u16* __restrict__ in, float* __restrict__ out, int64_t n) {
  GRID_LOOP(i, n) out[i] = bf16_to_f32(in[i]);
}

// out[r][0:c1] = A[r][:], out[r][c1:c1+c2] = B[r][:]
__global__ void concat_cols_kernel(const u16* __restrict__ A, const u16* __restrict__ Bm, u16* __restrict__ out,
                                   int64_t rows, int64_t c1, int64_t c2) {
  const int64_t w = c1 + c2, n = rows * w;
  GRID_LOOP(i, n) {
    const int64_t r = i / w, c = i - r * w;
    out[i] = c < c1 ? A[r * c1 + c] : Bm[r * c2 + (c - c1)];
  }
}

// A[r][:] = in[r][0:c], B[r][:] = in[r][c:2c] (either output nullable)
__global__ void split_cols_kernel(const float* __restrict__ in, float* __restrict__ A, float* __restrict__ Bm,
                                  int64_t rows, int64_t c) {
  const int64_t n = rows * 2 * c;
  GRID_LOOP(i, n) {
    const int64_t r = i / (2 * c), j = i - r * 2 * c;
    if (j < c) {
      if (A) A[r * c + j] = in[i];
    } else if (Bm) {
      Bm[r * c + j - c] = in[i];
    }
  }
}

// a = silu(g) * hh with gh = [g | hh] [T][2F]
__global__ void swiglu_fwd_kernel(const float* __restrict__ gh, float* __restrict__ a, int64_t T, int64_t F) {
  const int64_t n = T * F;
  GRID_LOOP(i, n) {
    const int64_t t = i / F, j = i - t * F;
    const float g = gh[t * 2 * F + j], hh = gh[t * 2 * F + F + j];
    a[i] = g / (1.0f + expf(-g)) * hh;
  }
}

// dg = da hh silu'(g), dhh = da silu(g), into [T][2F] (fp64 arithmetic, fp32 result)
__global__ void swiglu_bwd_kernel(const float* __restrict__ da, const float* __restrict__ gh, float* __restrict__ dgh,
                                  int64_t T, int64_t F) {
  const int64_t n = T * F;
  GRID_LOOP(i, n) {
    const int64_t t = i / F, j = i - t * F;
    const double g = gh[t * 2 * F + j], hh = gh[t * 2 * F + F + j], d = da[i];
    const double sg = 1.0 / (1.0 + exp(-g));
    dgh[t * 2 * F + j] = (float)(d * hh * sg * (1.0 + g * (1.0 - sg)));
    dgh[t * 2 * F + F + j] = (float)(d * g * sg);
  }
}

// out = a (bf16 or fp32) + b (fp32)
template <typename TA>
__global__ void add_kernel(const TA* __restrict__ a, const float* __restrict__ b, float* __restrict__ out, int64_t n) {
  GRID_LOOP(i, n) out[i] = load_f32(a, i) + b[i];
}
// the same, four elements per thread (16-byte aligned fp32 arrays, 8-byte aligned bf16)
__device__ __forceinline__ float4 load4f(const float* p, int64_t i) { return ((const float4*)p)[i]; }
__device__ __forceinline__ float4 load4f(const u16* p, int64_t i) {
  const uint2 v = ((const uint2*)p)[i];
  return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u), __uint_as_float(v.y << 16),
                     __uint_as_float(v.y & 0xFFFF0000u));
}
template <typename TA>
__global__ __launch_bounds__(256) void add4_kernel(const TA* __restrict__ a, const float* __restrict__ b,
                                                   float* __restrict__ out, int64_t n4) {
  GRID_LOOP(i, n4) {
    const float4 x = load4f(a, i), y = ((const float4*)b)[i];
    ((float4*)out)[i] = make_float4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
  }
}

// batched: grid (SUMSQ_BLOCKS, count); block b of job j sums x[i]^2 for i = b*256 + t, stepping
// by the grid, then the 4 waves in order; the final kernel folds the job's partials in a
// fixed tree
__global__ __launch_bounds__(256) void sumsq_batch_kernel(SumsqBatch b, double* __restrict__ part) {
  const SumsqJob j = b.job[blockIdx.y];
  double s = 0.0;
  if (j.x) {
    // 16-byte loads when the array allows them, then the scalar tail (fixed order per thread)
    const int64_t n4 = ((uintptr_t)j.x & 15) == 0 ? j.n / 4 : 0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)SUMSQ_BLOCKS * 256) {
      const float4 v = ((const float4*)j.x)[i];
      s += (double)v.x * v.x + (double)v.y * v.y + (double)v.z * v.z + (double)v.w * v.w;
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * 256 + threadIdx.x; i < j.n; i += (int64_t)SUMSQ_BLOCKS * 256) {
      const double v = j.x[i];
      s += v * v;
    }
  }
  __shared__ double red[4];
  s = wave_sum_f64(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) part[(int64_t)blockIdx.y * SUMSQ_BLOCKS + blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}
__global__ __launch_bounds__(256) void sumsq_batch_final(SumsqBatch b, const double* __restrict__ part) {
  const SumsqJob j = b.job[blockIdx.x];
  __shared__ double t[SUMSQ_BLOCKS];
  t[threadIdx.x] = j.x ? part[(int64_t)b.row[blockIdx.x] * SUMSQ_BLOCKS + threadIdx.x] : 0.0;
  __syncthreads();
  for (int o = SUMSQ_BLOCKS / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) t[threadIdx.x] += t[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) *j.out = j.x ? t[0] : (j.n == 1 ? 0.0 : __builtin_nan(""));
}


// ------------------------------------------------------------------------------------
static bool al(const void* p, int bytes);
static bool rows_ok(int B, int S);
bs_status launch_qkv_heads(const float* qkv, int B, int S, int H, int dh, u16* Q, u16* K, u16* V, hipStream_t st) {
  if (dh % 4 == 0 && al(qkv, 16) && al(Q, 8) && al(K, 8) && al(V, 8) && rows_ok(B, S))
    qkv_heads4_kernel<<<(unsigned)(B * S), 256, 0, st>>>((const float4*)qkv, S, H, dh, Q, K, V);
  else
    qkv_heads_kernel<<<blocks_for((int64_t)B * S * 3 * H * dh), 256, 0, st>>>(qkv, B, S, H, dh, Q, K, V);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
static bool al(const void* p, int bytes) { return ((uintptr_t)p & (uintptr_t)(bytes - 1)) == 0; }
// one block per token row (B S rows, at most 2^31 - 1)
static bool rows_ok(int B, int S) { return (int64_t)B * S > 0 && (int64_t)B * S < 2147483647LL; }
bs_status launch_heads_tokens_f32(const float* in, float* out, int B, int S, int H, int dh, bool to_tokens,
                                  hipStream_t st) {
  if (dh % 4 == 0 && al(in, 16) && al(out, 16) && rows_ok(B, S))
    heads_tokens4_kernel<float4><<<(unsigned)(B * S), 256, 0, st>>>((const float4*)in, (float4*)out, S, H, dh,
                                                                   to_tokens);
  else
    heads_tokens_kernel<float><<<blocks_for((int64_t)B * S * H * dh), 256, 0, st>>>(in, out, B, S, H, dh, to_tokens);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_heads_tokens_u8(const uint8_t* in, uint8_t* out, int B, int S, int H, int dh, hipStream_t st) {
  if (dh % 4 == 0 && al(in, 4) && al(out, 4) && rows_ok(B, S))
    heads_tokens4_kernel<uint32_t><<<(unsigned)(B * S), 256, 0, st>>>((const uint32_t*)in, (uint32_t*)out, S, H, dh,
                                                                     1);
  else
    heads_tokens_kernel<uint8_t><<<blocks_for((int64_t)B * S * H * dh), 256, 0, st>>>(in, out, B, S, H, dh, 1);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_dqkv_tokens(const float* dQ, const float* dK, const float* dV, float* out, int B, int S, int H,
                             int dh, hipStream_t st) {
  if (dh % 4 == 0 && al(dQ, 16) && al(dK, 16) && al(dV, 16) && al(out, 16) && rows_ok(B, S))
    dqkv_tokens4_kernel<<<(unsigned)(B * S), 256, 0, st>>>((const float4*)dQ, (const float4*)dK, (const float4*)dV,
                                                           (float4*)out, S, H, dh);
  else
    dqkv_tokens_kernel<<<blocks_for((int64_t)B * S * 3 * H * dh), 256, 0, st>>>(dQ, dK, dV, out, B, S, H, dh);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_bf16_to_f32(const u16* in, float* out, int64_t n, hipStream_t st) {
  if (n > 0) bf16_to_f32_kernel<<<blocks_for(n), 256, 0, st>>>(in, out, n);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_concat_cols(const u16* A, const u16* B, u16* out, int64_t rows, int64_t c1, int64_t c2,
                             hipStream_t st) {
  concat_cols_kernel<<<blocks_for(rows * (c1 + c2)), 256, 0, st>>>(A, B, out, rows, c1, c2);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_split_cols(const float* in, float* A, float* B, int64_t rows, int64_t c, hipStream_t st) {
  if (rows <= 0 || c <= 0 || (!A && !B)) return BS_OK;
  split_cols_kernel<<<blocks_for(rows * 2 * c), 256, 0, st>>>(in, A, B, rows, c);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_swiglu_fwd(const float* gh, float* a, int64_t T, int64_t F, hipStream_t st) {
  if (T > 0) swiglu_fwd_kernel<<<blocks_for(T * F), 256, 0, st>>>(gh, a, T, F);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_swiglu_bwd(const float* da, const float* gh, float* dgh, int64_t T, int64_t F, hipStream_t st) {
  if (T > 0) swiglu_bwd_kernel<<<blocks_for(T * F), 256, 0, st>>>(da, gh, dgh, T, F);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_add(const void* a, bs_dtype at, const float* b, float* out, int64_t n, hipStream_t st) {
  if (n <= 0) return BS_OK;
  const bool v4 = n % 4 == 0 && al(a, at == BS_F32 ? 16 : 8) && al(b, 16) && al(out, 16);
  if (v4 && at == BS_F32)
    add4_kernel<float><<<blocks_for(n / 4), 256, 0, st>>>((const float*)a, b, out, n / 4);
  else if (v4)
    add4_kernel<u16><<<blocks_for(n / 4), 256, 0, st>>>((const u16*)a, b, out, n / 4);
  else if (at == BS_F32)
    add_kernel<float><<<blocks_for(n), 256, 0, st>>>((const float*)a, b, out, n);
  else
    add_kernel<u16><<<blocks_for(n), 256, 0, st>>>((const u16*)a, b, out, n);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_sumsq_batch(const SumsqBatch& b, double* part, hipStream_t st) {
  if (b.count <= 0) return BS_OK;
  if (b.count > SUMSQ_MAX) return BS_EINVAL;
  // one partial-sum row per distinct (array, length): a reference read by several letters' rows
  // is summed once (same sum, same order)
  SumsqBatch u{}, f = b;
  for (int i = 0; i < b.count; ++i) {
    f.row[i] = -1;
    if (!b.job[i].x) continue;
    for (int k = 0; k < u.count && f.row[i] < 0; ++k)
      if (u.job[k].x == b.job[i].x && u.job[k].n == b.job[i].n) f.row[i] = k;
    if (f.row[i] < 0) {
      f.row[i] = u.count;
      u.job[u.count++] = b.job[i];
    }
  }
  if (u.count > 0) sumsq_batch_kernel<<<dim3(SUMSQ_BLOCKS, (unsigned)u.count), 256, 0, st>>>(u, part);
  sumsq_batch_final<<<(unsigned)f.count, SUMSQ_BLOCKS, 0, st>>>(f, part);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
