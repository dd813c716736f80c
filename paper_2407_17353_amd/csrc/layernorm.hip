// Scaled LayerNorm (Appendix C.2) and its input gradient with the dynamic
// rescale (the LayerNorm backward rescale of the experiments, Section 4).
//
// Forward: a mean-variance normalization is scale invariant up to its eps,
// so the data component X_d is normalized and the output gets scale 1:
//   xhat = (x - mean) / (std + eps),  y = xhat * gamma + beta,  cast(y).
// Backward: the gradient with respect to X_d, as the ScaledArray
// (dx, s_dy / s_x), then rebalanced by the amax rule and cast:
//   dx = (g - mean(g) - (c / std) mean(g * xhat)) / (std + eps),  g = dy * gamma,
//   c = x - mean; dgamma = sum_rows dy * xhat, dbeta = sum_rows dy.
//
// Row statistics: one wave per row; lane l takes the 16-column chunks l,
// l + 64, ... of the row, and the row sums are lane sums then a wave
// butterfly (no LDS, no barrier; fixed order, so reruns are bit-identical).
// Each pass over the row re-reads it (the later passes are served by the
// caches) so that a wave holds little and many rows are in flight. The
// forward's last pass writes y. The backward's statistic kernel also streams
// dy (twice: for mean(g), mean(g * xhat), then for dx's amax) and keeps, per
// row, the four numbers dx needs; its apply kernel is then a streaming pass over
// 32-row x 2048-column tiles that casts dx with the rescale the global amax
// gives and accumulates the tile's partial parameter gradients, which a last
// kernel sums over the row tiles in a fixed order.
#include "codec.h"
#include "ew_util.h"
#include "layernorm.h"

#include <stdlib.h>
#include <type_traits>

namespace scalify {

// f(std::integral_constant<int, I>), ..., up to N - 1 (compile-time indices).
template <int I, int N, typename F>
__device__ __forceinline__ void ln_static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    ln_static_for<I + 1, N>(f);
  }
}

constexpr int LN_THREADS = 256;   // 4 waves: 4 rows at a time
constexpr int LN_TILE_ROWS = 32;  // apply kernel: rows per workgroup
constexpr int LN_TILE_THREADS = 128;
constexpr int LN_TILE_COLS = 16 * LN_TILE_THREADS;

template <int F>
__device__ __forceinline__ void ln_chunk_f(const void* base, int64_t off, int valid,
                                           float (&v)[16]) {
  uint32_t c[16];
  if (valid >= 16) {
    load16<F>(base, off, c);
  } else {
    // ragged end of the row: element loads at clamped (valid) addresses
#pragma unroll
    for (int i = 0; i < 16; ++i) c[i] = load1<F>(base, off + (i < valid ? i : 0));
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] = i < valid ? decode_hw<F>(c[i]) : 0.0f;
}

// 16 values of a row from column n (columns >= D read as 0), format fmt.
__device__ __forceinline__ void ln_load16(int fmt, const void* base, int64_t off, int valid,
                                          float (&v)[16]) {
  if (fmt == kF16) ln_chunk_f<kF16>(base, off, valid, v);
  else if (fmt == kE4M3) ln_chunk_f<kE4M3>(base, off, valid, v);
  else if (fmt == kE5M2) ln_chunk_f<kE5M2>(base, off, valid, v);
  else ln_chunk_f<kF32>(base, off, valid, v);
}

__device__ __forceinline__ void ln_param16(const float* p, int n, int valid, float dflt,
                                           float (&v)[16]) {
  if (p == nullptr) {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = dflt;
  } else if (valid >= 16) {
    ln_chunk_f<kF32>(p, n, 16, v);
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = i < valid ? p[n + i] : dflt;
  }
}

__device__ __forceinline__ float wave_sum(float a) {
  for (int off = 32; off > 0; off >>= 1) a += __shfl_xor(a, off, 64);
  return a;
}

// Cast and store 16 values of one row at column n.
template <int OUTF>
__device__ __forceinline__ void ln_store16(void* out, int64_t off, int valid, const float (&y)[16],
                                           int shift, float scale, bool fast, bool sat) {
  uint32_t u[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) u[i] = __float_as_uint(y[i]);
  uint32_t w[8];
  encode16<OUTF>(u, shift, scale, fast, sat, w);
  if (valid >= 16) {
    store_words16<OUTF>(out, off, w);
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < valid) store1<OUTF>(out, off + i, word_code<OUTF>(w, i));
  }
}

__device__ __forceinline__ void ln_store_f32(float* q, int valid, const float (&y)[16]) {
  if (valid >= 16 && ((uintptr_t)q & 15u) == 0) {
#pragma unroll
    for (int h = 0; h < 4; ++h) *(u4*)(q + 4 * h) = u4{__float_as_uint(y[4 * h]), __float_as_uint(y[4 * h + 1]),
                                                         __float_as_uint(y[4 * h + 2]), __float_as_uint(y[4 * h + 3])};
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < valid) q[i] = y[i];
  }
}

// Mean and std of row r (fp32; lane sums over its chunks, then a wave
// butterfly): two passes over the row, the second one served by the caches.
template <int XF>
__device__ __forceinline__ void ln_row_stats(const LnParams& p, int64_t r, int lane, float& mu,
                                             float& sigma) {
  // (no FMA contraction: the fused multiply-adds are written out, the same
  // in the single-read and multi-pass kernels, so both round alike)
#pragma clang fp contract(off)
  const int nch = (p.D + 15) / 16;
  float s = 0.0f;
#pragma unroll 2
  for (int q = lane; q < nch; q += 64) {
    float v[16];
    ln_chunk_f<XF>(p.x, r * p.ldx + 16 * q, p.D - 16 * q, v);
#pragma unroll
    for (int i = 0; i < 16; ++i) s += v[i];  // columns >= D read as 0
  }
  mu = wave_sum(s) / (float)p.D;
  float t = 0.0f;
#pragma unroll 2
  for (int q = lane; q < nch; q += 64) {
    float v[16];
    const int valid = p.D - 16 * q;
    ln_chunk_f<XF>(p.x, r * p.ldx + 16 * q, valid, v);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float d = v[i] - mu;
      t = fmaf(i < valid ? d : 0.0f, d, t);  // (one rounding per term)
    }
  }
  sigma = sqrtf(wave_sum(t) / (float)p.D);
}

template <int XF, int OUTF>
__global__ __launch_bounds__(LN_THREADS) void ln_fwd_kernel(LnParams p) {
  // (no FMA contraction: the fused multiply-adds are written out, the same
  // in the single-read and multi-pass kernels, so both round alike)
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const bool sat = p.sat != 0;
  const int nch = (p.D + 15) / 16;
  if (blockIdx.x == 0 && threadIdx.x == 0) *p.out_scale = 1.0f;  // Appendix C.2: scale 1
#pragma unroll 1
  for (int64_t r = (int64_t)blockIdx.x * 4 + wave; r < p.R; r += (int64_t)gridDim.x * 4) {
    float mu, sigma;
    ln_row_stats<XF>(p, r, lane, mu, sigma);
    const float inv = 1.0f / (sigma + p.eps);
#pragma unroll 1
    for (int q = lane; q < nch; q += 64) {
      const int n = 16 * q;
      const int valid = p.D - n;
      float v[16], g[16], b[16], y[16];
      ln_chunk_f<XF>(p.x, r * p.ldx + n, valid, v);
      ln_param16(p.gamma, n, valid, 1.0f, g);
      ln_param16(p.beta, n, valid, 0.0f, b);
#pragma unroll
      for (int i = 0; i < 16; ++i) y[i] = fmaf((v[i] - mu) * inv, g[i], b[i]);
      if (p.pre_out) ln_store_f32(p.pre_out + r * (int64_t)p.D + n, valid, y);
      ln_store16<OUTF>(p.out, r * p.ldo + n, valid, y, 0, 1.0f, true, sat);
    }
  }
}

// The forward for rows of 2049 .. 4096 FP16 or FP8 elements, each row
// crossing HBM once: a wave holds its row's raw codes in registers (lane l
// the 16-element chunks l + 64 j, j < 4) and loads the next row of its
// stride while it computes this one (two buffers); gamma and beta sit in LDS
// for the workgroup's rows. The statistics and the output are computed in the
// order ln_row_stats and ln_fwd_kernel use, so the two kernels give the same
// bits. FULL: D = 4096, every chunk of every lane whole (no checks).
constexpr int LN_PIPE_NJ = 4;
constexpr int LN_PIPE_D = 1024 * LN_PIPE_NJ;

// An empty asm on the raw codes before each pass over them: the compiler then
// decodes them again instead of keeping every decoded value of the row
// alive across the passes (which would cost the occupancy).
template <int NJ, int W>
__device__ __forceinline__ void ln_opaque(uint32_t (&w)[NJ][W]) {
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int k = 0; k < W; ++k) asm volatile("" : "+v"(w[j][k]));
}

template <int XF>
__device__ __forceinline__ float ln_raw_decode(const uint32_t* w, int i) {
  if constexpr (XF == kF32) return __uint_as_float(w[i]);
  else if constexpr (XF == kF16) return decode_hw<kF16>((w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
  else return decode_hw<XF>((w[i >> 2] >> (8 * (i & 3))) & 0xFFu);
}

// Element I of a chunk's raw codes as fp32: an FP8 code is converted straight
// from its byte of the word (the conversion selects the byte).
template <int XF, int I>
__device__ __forceinline__ float ln_decode_at(const uint32_t* w) {
  if constexpr (XF == kE4M3) return __builtin_amdgcn_cvt_scalef32_f32_fp8(w[I >> 2], 1.0f, I & 3);
  else if constexpr (XF == kE5M2) return __builtin_amdgcn_cvt_scalef32_f32_bf8(w[I >> 2], 1.0f, I & 3);
  else return ln_raw_decode<XF>(w, I);
}

// The 16 elements of a chunk's raw codes as fp32 (exact), FP8 codes two per
// conversion (the packed form takes the low or the high 16 bits of a word).
template <int XF>
__device__ __forceinline__ void ln_decode16(const uint32_t* w, float (&x)[16]) {
  if constexpr (XF == kE4M3 || XF == kE5M2) {
    auto pk = [](uint32_t v, auto hi_tag) {
      if constexpr (XF == kE4M3)
        return __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(v, 1.0f, decltype(hi_tag)::value);
      else
        return __builtin_amdgcn_cvt_scalef32_pk_f32_bf8(v, 1.0f, decltype(hi_tag)::value);
    };
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const auto lo = pk(w[k], std::false_type{});
      const auto hi = pk(w[k], std::true_type{});
      x[4 * k] = lo[0];
      x[4 * k + 1] = lo[1];
      x[4 * k + 2] = hi[0];
      x[4 * k + 3] = hi[1];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = ln_raw_decode<XF>(w, i);
  }
}

// Dwords of a 16-element chunk of format F, and the chunk's raw codes at
// element e of base (valid elements, the rest zero: codes that decode to 0).
template <int F>
constexpr int ln_chunk_words() { return F == kF32 ? 16 : (F == kF16 ? 8 : 4); }

template <int F>
__device__ __forceinline__ void ln_load_raw(const void* base, int64_t e, int valid,
                                            uint32_t (&w)[ln_chunk_words<F>()]) {
  constexpr int W = ln_chunk_words<F>();
  constexpr int EPW = 16 / W;  // elements per dword
#pragma unroll
  for (int k = 0; k < W; ++k) w[k] = 0u;
  if (valid >= 16) {
#pragma unroll
    for (int h = 0; h < W / 4; ++h) {
      const u4 v = F == kF32 ? *((const u4*)((const uint32_t*)base + e) + h)
                             : (F == kF16 ? *((const u4*)((const uint16_t*)base + e) + h)
                                          : *((const u4*)((const uint8_t*)base + e) + h));
#pragma unroll
      for (int k = 0; k < 4; ++k) w[4 * h + k] = v[k];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < valid) w[i / EPW] |= load1<F>(base, e + i) << ((32 / EPW) * (i % EPW));
  }
}

template <int XF, int OUTF, bool FULL>
__global__ __launch_bounds__(LN_THREADS) void ln_fwd_pipe_kernel(LnParams p) {
  // (no FMA contraction: the fused multiply-adds are written out, the same
  // in the single-read and multi-pass kernels, so both round alike)
#pragma clang fp contract(off)
  constexpr int NJ = LN_PIPE_NJ;
  constexpr int WPC = XF == kF16 ? 8 : 4;  // dwords per 16-element chunk
  __shared__ __attribute__((aligned(16))) float s_g[LN_PIPE_D];
  __shared__ __attribute__((aligned(16))) float s_b[LN_PIPE_D];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const bool sat = p.sat != 0;
  const int D = p.D;
  const int nch = (D + 15) / 16;
  for (int e = threadIdx.x; e < 16 * nch; e += LN_THREADS) {
    s_g[e] = (p.gamma && e < D) ? p.gamma[e] : 1.0f;
    s_b[e] = (p.beta && e < D) ? p.beta[e] : 0.0f;
  }
  __syncthreads();
  if (blockIdx.x == 0 && threadIdx.x == 0) *p.out_scale = 1.0f;  // Appendix C.2: scale 1
  const int64_t stride = (int64_t)gridDim.x * 4;
  // raw codes of row r (zeros past D and for r >= R)
  auto load_row = [&](int64_t r, uint32_t (&w)[NJ][WPC]) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = lane + 64 * j;
      const int valid = D - 16 * q;
#pragma unroll
      for (int k = 0; k < WPC; ++k) w[j][k] = 0u;
      if (r < p.R && (FULL || q < nch)) {
        const int64_t e = r * p.ldx + 16 * q;
        if (FULL || valid >= 16) {
#pragma unroll
          for (int h = 0; h < WPC / 4; ++h) {
            const u4 v = XF == kF16 ? *((const u4*)((const uint16_t*)p.x + e) + h)
                                    : *((const u4*)((const uint8_t*)p.x + e) + h);
#pragma unroll
            for (int k = 0; k < 4; ++k) w[j][4 * h + k] = v[k];
          }
        } else {
          constexpr int EPW = XF == kF16 ? 2 : 4;  // elements per dword
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if (i < valid) w[j][i / EPW] |= load1<XF>(p.x, e + i) << ((32 / EPW) * (i % EPW));
        }
      }
    }
  };
  auto process = [&](int64_t r, uint32_t (&w)[NJ][WPC]) {
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (FULL || lane + 64 * j < nch) {
#pragma unroll
        for (int i = 0; i < 16; ++i) s += ln_raw_decode<XF>(w[j], i);  // columns >= D are 0
      }
    const float mu = wave_sum(s) / (float)D;
    float t = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = lane + 64 * j;
      if (FULL || q < nch) {
        const int valid = FULL ? 16 : D - 16 * q;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float d = ln_raw_decode<XF>(w[j], i) - mu;
          t = fmaf(i < valid ? d : 0.0f, d, t);  // (one rounding per term)
        }
      }
    }
    const float sigma = sqrtf(wave_sum(t) / (float)D);
    const float inv = 1.0f / (sigma + p.eps);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = lane + 64 * j;
      if (FULL || q < nch) {
        const int n = 16 * q;
        const int valid = FULL ? 16 : D - n;
        float y[16];
#pragma unroll
        for (int i = 0; i < 16; ++i)
          y[i] = fmaf((ln_raw_decode<XF>(w[j], i) - mu) * inv, s_g[n + i], s_b[n + i]);
        if (p.pre_out) ln_store_f32(p.pre_out + r * (int64_t)D + n, valid, y);
        ln_store16<OUTF>(p.out, r * p.ldo + n, valid, y, 0, 1.0f, true, sat);
      }
      // one chunk's gamma, beta and outputs at a time: bounded registers
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  uint32_t wa[NJ][WPC], wb[NJ][WPC];
  int64_t r = (int64_t)blockIdx.x * 4 + wave;
  load_row(r, wa);
#pragma unroll 1
  while (r < p.R) {
    load_row(r + stride, wb);
    process(r, wa);
    r += stride;
    if (r >= p.R) break;
    load_row(r + stride, wa);
    process(r, wb);
    r += stride;
  }
}

// Per-row numbers of the gradient (rowstats[r] = {mean, 1/(std+eps), mean(g),
// mean(g * xhat)/std or 0}), so that dx = (dy gamma - mean(g) - (x - mean) t) * inv.
// Both backward kernels evaluate it with this code and no contraction, so the
// apply kernel casts bit for bit the values whose amax the statistic measured.
__device__ __forceinline__ float ln_dx(float x, float dy, float gam, const float4& st) {
#pragma clang fp contract(off)
  const float g = dy * gam;
  return (g - st.z - (x - st.x) * st.w) * st.y;
}

template <int XF>
__global__ __launch_bounds__(LN_THREADS) void ln_bwd_stats_kernel(LnParams p) {
  // (no FMA contraction: the fused multiply-adds are written out, the same
  // in the single-read and multi-pass kernels, so both round alike)
#pragma clang fp contract(off)
  __shared__ float wmax[4];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nch = (p.D + 15) / 16;
  float lmax = 0.0f;
  float4* rowstats = (float4*)p.partial;
#pragma unroll 1
  for (int64_t r = (int64_t)blockIdx.x * 4 + wave; r < p.R; r += (int64_t)gridDim.x * 4) {
    float mu, sigma;
    ln_row_stats<XF>(p, r, lane, mu, sigma);
    const float inv = 1.0f / (sigma + p.eps);
    float sg = 0.0f, sgx = 0.0f;
#pragma unroll 1
    for (int q = lane; q < nch; q += 64) {
      const int n = 16 * q;
      const int valid = p.D - n;
      float v[16], d[16], gam[16];
      ln_chunk_f<XF>(p.x, r * p.ldx + n, valid, v);
      ln_load16(p.dy_fmt, p.dy, r * p.lddy + n, valid, d);
      ln_param16(p.gamma, n, valid, 1.0f, gam);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float g = i < valid ? d[i] * gam[i] : 0.0f;
        sg += g;
        sgx = fmaf(g, (v[i] - mu) * inv, sgx);
      }
    }
    sg = wave_sum(sg);
    sgx = wave_sum(sgx);
    float4 st;
    st.x = mu;
    st.y = inv;
    st.z = sg / (float)p.D;
    st.w = sigma > 0.0f ? (sgx / (float)p.D) / sigma : 0.0f;
    if (lane == 0) rowstats[r] = st;
#pragma unroll 1
    for (int q = lane; q < nch; q += 64) {
      const int n = 16 * q;
      const int valid = p.D - n;
      float v[16], d[16], gam[16], dx[16];
      ln_chunk_f<XF>(p.x, r * p.ldx + n, valid, v);
      ln_load16(p.dy_fmt, p.dy, r * p.lddy + n, valid, d);
      ln_param16(p.gamma, n, valid, 1.0f, gam);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        dx[i] = ln_dx(v[i], d[i], gam[i], st);
        if (i < valid) lmax = fmaxf(lmax, fabsf(dx[i]));  // fmaxf skips NaN
      }
      if (p.pre_out) ln_store_f32(p.pre_out + r * (int64_t)p.D + n, valid, dx);
    }
  }
  // amax of |dx|: wave butterfly, the four waves, one atomic max per workgroup
  for (int off = 32; off > 0; off >>= 1) lmax = fmaxf(lmax, __shfl_xor(lmax, off, 64));
  if (lane == 0) wmax[wave] = lmax;
  __syncthreads();
  if (threadIdx.x == 0)
    atomicMax(p.hdr, __float_as_uint(fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]))));
}

// The backward's statistics for rows of 2049 .. 4096 FP16 / FP8 elements,
// each row of x and dy read from HBM once: the wave holds both rows' raw
// codes in registers and loads the next rows of its stride while it computes
// these (two buffers); gamma sits in LDS. Same arithmetic, in the same order,
// as ln_bwd_stats_kernel.
// (three waves per SIMD: at most 170 VGPRs)
template <int XF, int DYF, bool FULL>
__global__ __launch_bounds__(LN_THREADS) __attribute__((amdgpu_waves_per_eu(3)))
void ln_bwd_stats_pipe_kernel(LnParams p) {
  // (no FMA contraction: the fused multiply-adds are written out, the same
  // in the single-read and multi-pass kernels, so both round alike)
#pragma clang fp contract(off)
  constexpr int NJ = LN_PIPE_NJ;
  constexpr int WX = XF == kF16 ? 8 : 4;    // dwords per 16-element chunk
  constexpr int WD = DYF == kF16 ? 8 : 4;
  __shared__ __attribute__((aligned(16))) float s_g[LN_PIPE_D];
  __shared__ float wmax[4];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int D = p.D;
  const int nch = (D + 15) / 16;
  for (int e = threadIdx.x; e < 16 * nch; e += LN_THREADS) s_g[e] = (p.gamma && e < D) ? p.gamma[e] : 1.0f;
  __syncthreads();
  float4* rowstats = (float4*)p.partial;
  const int64_t stride = (int64_t)gridDim.x * 4;
  auto load_chunks = [&](auto fmt_tag, const void* base, int64_t ld, int64_t r, auto& w) {
    constexpr int F = decltype(fmt_tag)::value;
    constexpr int W = F == kF16 ? 8 : 4;
    constexpr int EPW = F == kF16 ? 2 : 4;  // elements per dword
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = lane + 64 * j;
      const int valid = D - 16 * q;
#pragma unroll
      for (int k = 0; k < W; ++k) w[j][k] = 0u;
      if (r < p.R && (FULL || q < nch)) {
        const int64_t e = r * ld + 16 * q;
        if (FULL || valid >= 16) {
#pragma unroll
          for (int h = 0; h < W / 4; ++h) {
            const u4 v = F == kF16 ? *((const u4*)((const uint16_t*)base + e) + h)
                                   : *((const u4*)((const uint8_t*)base + e) + h);
#pragma unroll
            for (int k = 0; k < 4; ++k) w[j][4 * h + k] = v[k];
          }
        } else {
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if (i < valid) w[j][i / EPW] |= load1<F>(base, e + i) << ((32 / EPW) * (i % EPW));
        }
      }
    }
  };
  float lmax = 0.0f;
  auto process = [&](int64_t r, uint32_t (&wx)[NJ][WX], uint32_t (&wd)[NJ][WD]) {
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (FULL || lane + 64 * j < nch) {
#pragma unroll
        for (int i = 0; i < 16; ++i) s += ln_raw_decode<XF>(wx[j], i);
      }
    const float mu = wave_sum(s) / (float)D;
    ln_opaque(wx);
    float t = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = lane + 64 * j;
      if (FULL || q < nch) {
        const int valid = FULL ? 16 : D - 16 * q;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float d = ln_raw_decode<XF>(wx[j], i) - mu;
          t = fmaf(i < valid ? d : 0.0f, d, t);  // (one rounding per term)
        }
      }
    }
    const float sigma = sqrtf(wave_sum(t) / (float)D);
    const float inv = 1.0f / (sigma + p.eps);
    ln_opaque(wx);
    float sg = 0.0f, sgx = 0.0f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = lane + 64 * j;
      if (FULL || q < nch) {
        const int n = 16 * q;
        const int valid = FULL ? 16 : D - n;
        ln_static_for<0, 16>([&](auto I) {
          constexpr int i = decltype(I)::value;
          const float g = i < valid ? ln_decode_at<DYF, i>(wd[j]) * s_g[n + i] : 0.0f;
          sg += g;
          sgx = fmaf(g, (ln_decode_at<XF, i>(wx[j]) - mu) * inv, sgx);
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    sg = wave_sum(sg);
    sgx = wave_sum(sgx);
    float4 st;
    st.x = mu;
    st.y = inv;
    st.z = sg / (float)D;
    st.w = sigma > 0.0f ? (sgx / (float)D) / sigma : 0.0f;
    if (lane == 0) rowstats[r] = st;
    ln_opaque(wx);
    ln_opaque(wd);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = lane + 64 * j;
      if (FULL || q < nch) {
        const int n = 16 * q;
        const int valid = FULL ? 16 : D - n;
        float dx[16];
        ln_static_for<0, 16>([&](auto I) {
          constexpr int i = decltype(I)::value;
          dx[i] = ln_dx(ln_decode_at<XF, i>(wx[j]), ln_decode_at<DYF, i>(wd[j]), s_g[n + i], st);
          if (i < valid) lmax = fmaxf(lmax, fabsf(dx[i]));  // fmaxf skips NaN
        });
        if (p.pre_out) ln_store_f32(p.pre_out + r * (int64_t)D + n, valid, dx);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using XT = std::integral_constant<int, XF>;
  using DT = std::integral_constant<int, DYF>;
  uint32_t xa[NJ][WX], xb[NJ][WX], da[NJ][WD], db[NJ][WD];
  int64_t r = (int64_t)blockIdx.x * 4 + wave;
  load_chunks(XT{}, p.x, p.ldx, r, xa);
  load_chunks(DT{}, p.dy, p.lddy, r, da);
#pragma unroll 1
  while (r < p.R) {
    load_chunks(XT{}, p.x, p.ldx, r + stride, xb);
    load_chunks(DT{}, p.dy, p.lddy, r + stride, db);
    process(r, xa, da);
    r += stride;
    if (r >= p.R) break;
    load_chunks(XT{}, p.x, p.ldx, r + stride, xa);
    load_chunks(DT{}, p.dy, p.lddy, r + stride, da);
    process(r, xb, db);
    r += stride;
  }
  // amax of |dx|: wave butterfly, the four waves, one atomic max per workgroup
  for (int off = 32; off > 0; off >>= 1) lmax = fmaxf(lmax, __shfl_xor(lmax, off, 64));
  if (lane == 0) wmax[wave] = lmax;
  __syncthreads();
  if (threadIdx.x == 0)
    atomicMax(p.hdr, __float_as_uint(fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]))));
}

// Tile (row block blockIdx.y of LN_TILE_ROWS rows, column block blockIdx.x of
// LN_TILE_COLS columns): dx recomputed from the row numbers, cast with the
// rescale, and the tile's partial parameter gradients.
template <int XF, int DYF, int OUTF>
__global__ __launch_bounds__(LN_TILE_THREADS) void ln_bwd_apply_kernel(LnParams p) {
  const int e_in = (int)p.hdr[1];
  int e_r = 0;
  if (p.mode == 1) e_r = rescale_exponent(p.hdr[0], p.target);
  const int e_out = clamp_e8m0(e_in + e_r);
  const int shift = e_out - e_in;
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
    *p.out_scale = pow2_float(e_out);
    if (p.amax_out) *p.amax_out = __uint_as_float(p.hdr[0]);
  }
  const bool sat = p.sat != 0;
  const bool fast = shift >= kFastShiftMinSub && shift <= kFastShiftMax;
  const float scale = fast ? pow2_float(shift) : 1.0f;
  const int n = (int)blockIdx.x * LN_TILE_COLS + 16 * (int)threadIdx.x;
  const int valid = p.D - n;
  const float4* rowstats = (const float4*)p.partial;
  const int64_t dp = layernorm_param_stride(p.D);
  float* part = p.partial + 4 * p.R + (int64_t)blockIdx.y * 2 * dp;
  if (valid <= 0) return;
  float gam[16], pg[16], pb[16];
  ln_param16(p.gamma, n, valid, 1.0f, gam);
#pragma unroll
  for (int i = 0; i < 16; ++i) pg[i] = pb[i] = 0.0f;
  const int64_t r0 = (int64_t)blockIdx.y * LN_TILE_ROWS;
  const int64_t r1 = r0 + LN_TILE_ROWS < p.R ? r0 + LN_TILE_ROWS : p.R;
  // The rows' raw codes go through a ring of PF slots: slot k holds row
  // rb + k while it is computed and then receives row rb + k + PF, so PF
  // rows' loads are in flight while one is computed (the per-row sums keep
  // their row order).
  constexpr int PF = 4;
  uint32_t rx[PF][ln_chunk_words<XF>()], rd[PF][ln_chunk_words<DYF>()];
#pragma unroll
  for (int k = 0; k < PF; ++k)
    if (r0 + k < r1) {
      ln_load_raw<XF>(p.x, (r0 + k) * p.ldx + n, valid, rx[k]);
      ln_load_raw<DYF>(p.dy, (r0 + k) * p.lddy + n, valid, rd[k]);
    }
#pragma unroll 1
  for (int64_t rb = r0; rb < r1; rb += PF) {
    ln_static_for<0, PF>([&](auto K) {
      constexpr int k = decltype(K)::value;
      const int64_t r = rb + k;
      if (r < r1) {
        const float4 st = rowstats[r];
        float dx[16];
        float xv[16], dv[16];
        ln_decode16<XF>(rx[k], xv);
        ln_decode16<DYF>(rd[k], dv);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float x = xv[i], d = dv[i];
          dx[i] = ln_dx(x, d, gam[i], st);
          pg[i] += d * ((x - st.x) * st.y);
          pb[i] += d;
        }
        ln_store16<OUTF>(p.out, r * p.ldo + n, valid, dx, shift, scale, fast, sat);
        if (r + PF < r1) {
          ln_load_raw<XF>(p.x, (r + PF) * p.ldx + n, valid, rx[k]);
          ln_load_raw<DYF>(p.dy, (r + PF) * p.lddy + n, valid, rd[k]);
        }
      }
    });
  }
  if (p.dgamma || p.dbeta) {
    ln_store_f32(part + n, valid, pg);
    ln_store_f32(part + dp + n, valid, pb);
  }
}

// dgamma[j], dbeta[j] = fixed-order sums of the row tiles' partials: a
// workgroup covers 64 columns; its LN_PARAM_WAVES waves sum interleaved
// shares of the tiles (wave w: tiles w, w + LN_PARAM_WAVES, ...), then wave
// 0 adds the wave sums pairwise in a fixed tree. (Few columns, many tiles:
// the waves of a workgroup keep more of the tiles' loads in flight.)
constexpr int LN_PARAM_WAVES = 16;

__global__ __launch_bounds__(64 * LN_PARAM_WAVES) void ln_params_kernel(const float* part, int tiles,
                                                                        int D, float* dgamma,
                                                                        float* dbeta) {
  __shared__ float red[2][LN_PARAM_WAVES][64];
  const int c = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + c;
  const int64_t dp = layernorm_param_stride(D);
  float g = 0.0f, b = 0.0f;
  if (j < D) {
#pragma unroll 8
    for (int k = w; k < tiles; k += LN_PARAM_WAVES) {
      g += part[(int64_t)k * 2 * dp + j];
      b += part[(int64_t)k * 2 * dp + dp + j];
    }
  }
  red[0][w][c] = g;
  red[1][w][c] = b;
  __syncthreads();
  if (w == 0 && j < D) {
    float sg[LN_PARAM_WAVES], sb[LN_PARAM_WAVES];
#pragma unroll
    for (int i = 0; i < LN_PARAM_WAVES; ++i) {
      sg[i] = red[0][i][c];
      sb[i] = red[1][i][c];
    }
#pragma unroll
    for (int h = 1; h < LN_PARAM_WAVES; h *= 2)
#pragma unroll
      for (int i = 0; i < LN_PARAM_WAVES; i += 2 * h) {
        sg[i] += sg[i + h];
        sb[i] += sb[i + h];
      }
    if (dgamma) dgamma[j] = sg[0];
    if (dbeta) dbeta[j] = sb[0];
  }
}

// hdr[0] = 0 (amax), hdr[1] = e(s_dy) - e(s_x): the gradient's scale exponent.
__global__ void ln_bwd_prologue_kernel(uint32_t* hdr, const float* s_dy, const float* s_x) {
  if (threadIdx.x == 0) {
    hdr[0] = 0u;
    hdr[1] = (uint32_t)(pow2_exponent(s_dy) - pow2_exponent(s_x));
  }
}

static int row_grid(int64_t R) {
  const int64_t b = (R + 3) / 4;
  return (int)(b < 1 ? 1 : (b > 8192 ? 8192 : b));
}

int64_t layernorm_row_tiles(int64_t R) {
  const int64_t t = (R + LN_TILE_ROWS - 1) / LN_TILE_ROWS;
  return t < 1 ? 1 : t;
}

int64_t layernorm_ws_floats(int64_t R, int64_t D) {
  return 4 * R + layernorm_row_tiles(R) * 2 * layernorm_param_stride(D);
}

// Workgroups of the pipelined kernels: per_cu per CU (as many as their
// registers let run at once), each wave walking rows with the grid's stride.
static int pipe_grid(int64_t R, int per_cu) {
  static int cus = 0;  // (a benign race: every thread computes the same value)
  if (cus <= 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus = n;
  }
  const int64_t need = (R + 3) / 4;
  const int64_t g = (int64_t)per_cu * cus;
  return (int)(need < 1 ? 1 : (need < g ? need : g));
}

// The single-read kernels unless SCALIFY_LN_SINGLE_READ=0 (read at each
// call), which keeps the multi-pass ones for every width.
static bool single_read_enabled() {
  const char* v = getenv("SCALIFY_LN_SINGLE_READ");
  return !(v && v[0] == '0' && v[1] == 0);
}

template <int XF>
static void launch_fwd_xf(const LnParams& p, int out_dtype, hipStream_t s) {
  const dim3 b(LN_THREADS);
  if constexpr (XF != kF32) {
    if (p.D > LN_PIPE_D / 2 && p.D <= LN_PIPE_D && single_read_enabled()) {
      const dim3 g(pipe_grid(p.R, 3));
      if (p.D == LN_PIPE_D) {
        if (out_dtype == kE4M3) hipLaunchKernelGGL((ln_fwd_pipe_kernel<XF, kE4M3, true>), g, b, 0, s, p);
        else if (out_dtype == kE5M2) hipLaunchKernelGGL((ln_fwd_pipe_kernel<XF, kE5M2, true>), g, b, 0, s, p);
        else hipLaunchKernelGGL((ln_fwd_pipe_kernel<XF, kF16, true>), g, b, 0, s, p);
      } else {
        if (out_dtype == kE4M3) hipLaunchKernelGGL((ln_fwd_pipe_kernel<XF, kE4M3, false>), g, b, 0, s, p);
        else if (out_dtype == kE5M2) hipLaunchKernelGGL((ln_fwd_pipe_kernel<XF, kE5M2, false>), g, b, 0, s, p);
        else hipLaunchKernelGGL((ln_fwd_pipe_kernel<XF, kF16, false>), g, b, 0, s, p);
      }
      return;
    }
  }
  const dim3 g(row_grid(p.R));
  if (out_dtype == kE4M3) hipLaunchKernelGGL((ln_fwd_kernel<XF, kE4M3>), g, b, 0, s, p);
  else if (out_dtype == kE5M2) hipLaunchKernelGGL((ln_fwd_kernel<XF, kE5M2>), g, b, 0, s, p);
  else hipLaunchKernelGGL((ln_fwd_kernel<XF, kF16>), g, b, 0, s, p);
}

hipError_t launch_layernorm_fwd(const LnParams& p, int out_dtype, hipStream_t s) {
  if (p.x_fmt == kF16) launch_fwd_xf<kF16>(p, out_dtype, s);
  else if (p.x_fmt == kF32) launch_fwd_xf<kF32>(p, out_dtype, s);
  else if (p.x_fmt == kE4M3) launch_fwd_xf<kE4M3>(p, out_dtype, s);
  else launch_fwd_xf<kE5M2>(p, out_dtype, s);
  return hipGetLastError();
}

template <int XF, int DYF>
static void launch_apply(const LnParams& p, int out_dtype, dim3 g, dim3 b, hipStream_t s) {
  if (out_dtype == kE4M3) hipLaunchKernelGGL((ln_bwd_apply_kernel<XF, DYF, kE4M3>), g, b, 0, s, p);
  else if (out_dtype == kE5M2) hipLaunchKernelGGL((ln_bwd_apply_kernel<XF, DYF, kE5M2>), g, b, 0, s, p);
  else hipLaunchKernelGGL((ln_bwd_apply_kernel<XF, DYF, kF16>), g, b, 0, s, p);
}

template <int XF>
static void launch_apply_x(const LnParams& p, int out_dtype, dim3 g, dim3 b, hipStream_t s) {
  if (p.dy_fmt == kF16) launch_apply<XF, kF16>(p, out_dtype, g, b, s);
  else if (p.dy_fmt == kF32) launch_apply<XF, kF32>(p, out_dtype, g, b, s);
  else if (p.dy_fmt == kE4M3) launch_apply<XF, kE4M3>(p, out_dtype, g, b, s);
  else launch_apply<XF, kE5M2>(p, out_dtype, g, b, s);
}

template <int XF, int DYF>
static void launch_stats_pipe(const LnParams& p, hipStream_t s) {
  const dim3 g(pipe_grid(p.R, 3)), b(LN_THREADS);
  if (p.D == LN_PIPE_D) hipLaunchKernelGGL((ln_bwd_stats_pipe_kernel<XF, DYF, true>), g, b, 0, s, p);
  else hipLaunchKernelGGL((ln_bwd_stats_pipe_kernel<XF, DYF, false>), g, b, 0, s, p);
}

template <int XF>
static void launch_stats_pipe_x(const LnParams& p, hipStream_t s) {
  if (p.dy_fmt == kF16) launch_stats_pipe<XF, kF16>(p, s);
  else if (p.dy_fmt == kE4M3) launch_stats_pipe<XF, kE4M3>(p, s);
  else launch_stats_pipe<XF, kE5M2>(p, s);
}

hipError_t launch_layernorm_bwd(const LnParams& p, const float* s_dy, const float* s_x,
                                int out_dtype, hipStream_t s) {
  hipLaunchKernelGGL(ln_bwd_prologue_kernel, dim3(1), dim3(64), 0, s, p.hdr, s_dy, s_x);
  if (p.R > 0 && p.x_fmt != kF32 && p.dy_fmt != kF32 && p.D > LN_PIPE_D / 2 && p.D <= LN_PIPE_D &&
      single_read_enabled()) {
    if (p.x_fmt == kF16) launch_stats_pipe_x<kF16>(p, s);
    else if (p.x_fmt == kE4M3) launch_stats_pipe_x<kE4M3>(p, s);
    else launch_stats_pipe_x<kE5M2>(p, s);
  } else if (p.R > 0) {
    const dim3 g(row_grid(p.R)), b(LN_THREADS);
    if (p.x_fmt == kF16) hipLaunchKernelGGL((ln_bwd_stats_kernel<kF16>), g, b, 0, s, p);
    else if (p.x_fmt == kF32) hipLaunchKernelGGL((ln_bwd_stats_kernel<kF32>), g, b, 0, s, p);
    else if (p.x_fmt == kE4M3) hipLaunchKernelGGL((ln_bwd_stats_kernel<kE4M3>), g, b, 0, s, p);
    else hipLaunchKernelGGL((ln_bwd_stats_kernel<kE5M2>), g, b, 0, s, p);
  }
  // The apply kernel also writes the output scale: at least one workgroup.
  const int64_t tiles = layernorm_row_tiles(p.R);
  const int cols = (p.D + LN_TILE_COLS - 1) / LN_TILE_COLS;
  const dim3 ga(cols < 1 ? 1 : cols, (unsigned)tiles);
  const dim3 ba(LN_TILE_THREADS);
  if (p.x_fmt == kF16) launch_apply_x<kF16>(p, out_dtype, ga, ba, s);
  else if (p.x_fmt == kF32) launch_apply_x<kF32>(p, out_dtype, ga, ba, s);
  else if (p.x_fmt == kE4M3) launch_apply_x<kE4M3>(p, out_dtype, ga, ba, s);
  else launch_apply_x<kE5M2>(p, out_dtype, ga, ba, s);
  if ((p.dgamma || p.dbeta) && p.D > 0)
    hipLaunchKernelGGL(ln_params_kernel, dim3((p.D + 63) / 64), dim3(64 * LN_PARAM_WAVES), 0, s,
                       p.partial + 4 * p.R,
                       (int)tiles, p.D, p.dgamma, p.dbeta);
  return hipGetLastError();
}

}  // namespace scalify
