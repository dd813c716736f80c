// HBM-bound kernels of the scaled-matmul epilogue and of the standalone
// ScaledArray operations:
//   * prologue: clears the amax word and snapshots input scale exponents;
//   * epilogue_cast: the grid-wide dependent half of the fused dynamic
//     rescale (Section 3.3): reads the global amax, derives the power-of-two
//     rescale exponent (rounded down), writes the output scale, and casts the
//     GEMM's pre-cast intermediate with round-to-nearest-even;
//   * amax: |x| max of an existing ScaledArray's data, as an integer max over
//     magnitude keys (no decode in the hot loop);
//   * elementwise: rebalance / set_scaling / cast of a ScaledArray's data.
// Every kernel moves 16 elements per thread per iteration with 128-bit
// loads; the cast kernel walks rows of the intermediate, the amax and
// elementwise kernels walk 1024-element blocks (layout below).
#include "codec.h"
#include "ew_util.h"
#include "kernels.h"

namespace scalify {

constexpr int EW_THREADS = 256;

__global__ void prologue_kernel(uint32_t* hdr, const float* s0, const float* s1) {
  if (threadIdx.x == 0) {
    hdr[0] = 0u;
    hdr[1] = (uint32_t)(pow2_exponent(s0) + pow2_exponent(s1));
  }
}

hipError_t launch_prologue(uint32_t* hdr, const float* s0, const float* s1, hipStream_t s) {
  hipLaunchKernelGGL(prologue_kernel, dim3(1), dim3(64), 0, s, hdr, s0, s1);
  return hipGetLastError();
}

// Matmul prologue: the scale exponent e_w of the pre-cast value (scaled add
// rule of Algorithm 3 with a residual) and, for the delayed rescale
// (Section 3.3), the output scale from the statistic an earlier call
// recorded, or without a rescale the propagated scale itself, so that the
// GEMM can cast directly; clears the statistic and the single-pass barrier.
__global__ void matmul_prologue_kernel(uint32_t* hdr, MatmulPrologue q) {
  if (threadIdx.x == 0) {
    const int e_ab = pow2_exponent(q.s0) + pow2_exponent(q.s1);
    int e_w = e_ab, e_cc = q.e_c;
    if (q.residual) {
      // sqrt(2^(2 e_p) + 2^(2 e_q)) rounded down to a power of two is the
      // larger of the two scales.
      const int e_q = pow2_exponent(q.s_res);
      e_w = max(e_ab + q.e_c, e_q);
      e_cc = 0;
      hdr[3] = (uint32_t)(e_ab - e_w);
      hdr[4] = (uint32_t)(e_q - e_w);
    }
    hdr[0] = 0u;
    hdr[1] = (uint32_t)e_w;
    hdr[5] = hdr[6] = hdr[7] = 0u;
    if (q.direct) {
      // |statistic| of an earlier call (delayed rescale), or none (e_r = 0)
      const uint32_t stat = q.amax_in ? __float_as_uint(*q.amax_in) & 0x7FFFFFFFu : 0u;
      const int e_r = rescale_exponent(stat, q.target);  // 0 for 0, Inf, NaN
      const int e_out = clamp_e8m0(e_w + e_cc + e_r);
      hdr[2] = (uint32_t)(e_out - e_w);
      *q.out_scale = pow2_float(e_out);
    }
  }
}

hipError_t launch_matmul_prologue(uint32_t* hdr, const MatmulPrologue& q, hipStream_t s) {
  hipLaunchKernelGGL(matmul_prologue_kernel, dim3(1), dim3(64), 0, s, hdr, q);
  return hipGetLastError();
}

__global__ void finalize_amax_kernel(const uint32_t* hdr, int e_c, float* amax_out) {
  if (threadIdx.x == 0) *amax_out = __uint_as_float(hdr[0]) * pow2_float(-e_c);
}

hipError_t launch_finalize_amax(const uint32_t* hdr, int e_c, float* amax_out, hipStream_t s) {
  hipLaunchKernelGGL(finalize_amax_kernel, dim3(1), dim3(64), 0, s, hdr, e_c, amax_out);
  return hipGetLastError();
}

// ---------------------------------------------------------------- GEMM epilogue cast

// NT: the 16-bit intermediate is larger than the last-level cache (MALL), so it is
// streamed from HBM with nontemporal loads and the codes written with
// nontemporal stores, which keeps the cache from thrashing; a smaller
// intermediate, just written by the GEMM, is still in the MALL and is read
// through it.
template <int INTER32, int OUTF, bool NT>
__global__ __launch_bounds__(EW_THREADS) void epilogue_cast_kernel(EpilogueParams p) {
  const uint32_t amax_raw = p.hdr[0];  // max |w| bits
  const int e_ab = (int)p.hdr[1];      // e_w
  int e_r = 0;
  if (p.mode == 1 && amax_raw != 0u && amax_raw < 0x7F800000u)
    e_r = floor_log2_bits(amax_raw) - p.e_c - p.target;
  const int e_out = clamp_e8m0(e_ab + p.e_c + e_r);
  const int shift = e_out - e_ab;  // data' = acc * 2^-shift
  const bool sat = p.sat != 0;
  const bool fast = shift >= kFastShiftMinSub && shift <= kFastShiftMax;
  const float scale = fast ? pow2_float(shift) : 1.0f;
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
    *p.out_scale = pow2_float(e_out);
    if (p.amax_out) *p.amax_out = __uint_as_float(amax_raw) * pow2_float(-p.e_c);
  }
  // 2-D grid: blockIdx.y walks rows, x-threads walk 16-element chunks.
  const int cpr = (p.N + 15) / 16;
  for (int m = blockIdx.y; m < p.M; m += gridDim.y) {
    for (int ch = blockIdx.x * EW_THREADS + threadIdx.x; ch < cpr; ch += gridDim.x * EW_THREADS) {
      const int n = ch * 16;
      uint32_t c[16];
      const int64_t e = (int64_t)m * p.ldw + n;
      if (INTER32) {
        if constexpr (NT) {
          const u4* q = (const u4*)((const uint32_t*)p.inter + e);
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            const u4 v = __builtin_nontemporal_load(q + h);
#pragma unroll
            for (int i = 0; i < 4; ++i) c[4 * h + i] = v[i];
          }
        } else {
          load16<kF32>(p.inter, e, c);
        }
      } else {
        if constexpr (NT) {
          const u4* q = (const u4*)((const uint16_t*)p.inter + e);
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const u4 v = __builtin_nontemporal_load(q + h);
#pragma unroll
            for (int i = 0; i < 8; ++i) c[8 * h + i] = (v[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
          }
        } else {
          load16<kF16>(p.inter, e, c);  // 16-bit containers
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) c[i] <<= 16;
      }
      uint32_t w[8];
      encode16<OUTF>(c, shift, scale, fast, sat, w);
      if (n + 16 <= p.N) {
        if constexpr (NT && OUTF == kF16) {
          u4* q = (u4*)((uint16_t*)p.out + (int64_t)m * p.ldc + n);
          __builtin_nontemporal_store(u4{w[0], w[1], w[2], w[3]}, q);
          __builtin_nontemporal_store(u4{w[4], w[5], w[6], w[7]}, q + 1);
        } else if constexpr (NT) {
          __builtin_nontemporal_store(u4{w[0], w[1], w[2], w[3]},
                                      (u4*)((uint8_t*)p.out + (int64_t)m * p.ldc + n));
        } else {
          store_words16<OUTF>(p.out, (int64_t)m * p.ldc + n, w);
        }
      } else {
        for (int i = 0; i < 16; ++i)
          if (n + i < p.N) store1<OUTF>(p.out, (int64_t)m * p.ldc + n + i, word_code<OUTF>(w, i));
      }
    }
  }
}


// 16-bit intermediates above this size no longer sit in the 256 MiB MALL
// after the GEMM has written them. Measured (cast kernel alone): nontemporal
// access takes a 384 MiB intermediate from 123.5 to 95 us and a 512 MiB one
// from 182 to 145 us, but a 128 MiB one from 32 to 34 us; for the fp32
// intermediate of FP16 outputs it made 8192 x 8192 slower (90 -> 110 us), so
// that one is always read through the caches.
constexpr int64_t kStreamingBytes = (int64_t)192 << 20;

template <bool NT>
void launch_cast(const EpilogueParams& p, int inter32, int out_dtype, dim3 g, dim3 b,
                 hipStream_t s) {
  if (inter32 && out_dtype == kF16) {
    hipLaunchKernelGGL((epilogue_cast_kernel<1, kF16, NT>), g, b, 0, s, p);
  } else if (inter32 && out_dtype == kE4M3) {
    hipLaunchKernelGGL((epilogue_cast_kernel<1, kE4M3, NT>), g, b, 0, s, p);
  } else if (inter32) {
    hipLaunchKernelGGL((epilogue_cast_kernel<1, kE5M2, NT>), g, b, 0, s, p);
  } else if (out_dtype == kE4M3) {
    hipLaunchKernelGGL((epilogue_cast_kernel<0, kE4M3, NT>), g, b, 0, s, p);
  } else {
    hipLaunchKernelGGL((epilogue_cast_kernel<0, kE5M2, NT>), g, b, 0, s, p);
  }
}

hipError_t launch_epilogue_cast(const EpilogueParams& p, int inter32, int out_dtype,
                                hipStream_t s) {
  const int cpr = (p.N + 15) / 16;
  const int gx = (cpr + EW_THREADS - 1) / EW_THREADS;
  const int gy = p.M < 1 ? 1 : (p.M > 65535 ? 65535 : p.M);
  const dim3 g(gx < 1 ? 1 : gx, gy), b(EW_THREADS);
  const int64_t inter_bytes = (int64_t)p.M * p.ldw * 2;
  if (!inter32 && inter_bytes > kStreamingBytes)
    launch_cast<true>(p, inter32, out_dtype, g, b, s);
  else
    launch_cast<false>(p, inter32, out_dtype, g, b, s);
  return hipGetLastError();
}

// ---------------------------------------------------------------- amax / elementwise
//
// Block layout of the streaming kernels: a block is 1024 consecutive
// elements, read by one wave as W 16-byte words per lane (W = 4 for fp32, 2
// for FP16, 1 for FP8): word w of lane l is word 64 w + l of the block, so
// every load instruction of the wave reads 1 KiB of consecutive bytes, and
// a lane's 16 elements are the EPW = 16 / W elements of each of its words.
// Waves walk the blocks with a stride of the whole grid, two blocks per
// iteration (2 W loads in flight per lane); the last partial block is done
// element by element by the first workgroup.
constexpr int EW_GRID = 2048;  // workgroups of 4 waves: 8 per CU

template <int F>
struct BlockLayout {
  static constexpr int ESZ = F == kF32 ? 4 : (F == kF16 ? 2 : 1);
  static constexpr int EPW = 16 / ESZ;  // elements per 16-byte word
  static constexpr int W = 16 / EPW;    // words per lane and block
};

// Load block b's words of this lane (raw 16-byte words).
template <int F>
__device__ __forceinline__ void load_block(const void* in, int64_t b, int lane,
                                           u4 (&w)[BlockLayout<F>::W]) {
  constexpr int W = BlockLayout<F>::W;
  const u4* q = (const u4*)in + b * (64 * W) + lane;
#pragma unroll
  for (int k = 0; k < W; ++k) w[k] = q[64 * k];
}

// The lane's 16 elements of a block as codes (or fp32 bits), word by word.
template <int F>
__device__ __forceinline__ void unpack_block(const u4 (&w)[BlockLayout<F>::W], uint32_t (&c)[16]) {
  constexpr int W = BlockLayout<F>::W, EPW = BlockLayout<F>::EPW;
#pragma unroll
  for (int k = 0; k < W; ++k)
#pragma unroll
    for (int i = 0; i < EPW; ++i) {
      const uint32_t word = w[k][i * 4 / EPW];
      if constexpr (F == kF32) c[k * EPW + i] = word;
      else if constexpr (F == kF16) c[k * EPW + i] = (word >> (16 * (i & 1))) & 0xFFFFu;
      else c[k * EPW + i] = (word >> (8 * (i & 3))) & 0xFFu;
    }
}

template <int F>
__global__ __launch_bounds__(EW_THREADS) void amax_kernel(const void* in, int64_t n,
                                                           uint32_t* hdr) {
  using L = BlockLayout<F>;
  __shared__ uint32_t red[EW_THREADS / 64];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (EW_THREADS / 64) + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * (EW_THREADS / 64);
  const int64_t nb = n / 1024;
  uint32_t kmax = 0;
  int64_t b = wave;
  for (; b + waves < nb; b += 2 * waves) {
    u4 w0[L::W], w1[L::W];
    load_block<F>(in, b, lane, w0);
    load_block<F>(in, b + waves, lane, w1);
    uint32_t c[16];
    unpack_block<F>(w0, c);
#pragma unroll
    for (int i = 0; i < 16; ++i) kmax = max(kmax, magnitude_key<F>(c[i]));
    unpack_block<F>(w1, c);
#pragma unroll
    for (int i = 0; i < 16; ++i) kmax = max(kmax, magnitude_key<F>(c[i]));
  }
  if (b < nb) {
    u4 w0[L::W];
    load_block<F>(in, b, lane, w0);
    uint32_t c[16];
    unpack_block<F>(w0, c);
#pragma unroll
    for (int i = 0; i < 16; ++i) kmax = max(kmax, magnitude_key<F>(c[i]));
  }
  if (blockIdx.x == 0)
    for (int64_t e = nb * 1024 + threadIdx.x; e < n; e += EW_THREADS)
      kmax = max(kmax, magnitude_key<F>(load1<F>(in, e)));
  for (int off = 32; off > 0; off >>= 1) kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, off, 64));
  if (lane == 0) red[threadIdx.x >> 6] = kmax;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t k = red[0];
    for (int w = 1; w < EW_THREADS / 64; ++w) k = max(k, red[w]);
    atomicMax(hdr, to_bits<F>(k));
  }
}

static int ew_grid(int64_t n) {
  const int64_t waves = (n + 1023) / 1024;  // one wave per block at most
  int64_t g = (waves + EW_THREADS / 64 - 1) / (EW_THREADS / 64);
  if (g < 1) g = 1;
  if (g > EW_GRID) g = EW_GRID;
  return (int)g;
}

hipError_t launch_amax(const void* in, int in_dtype, int64_t n, uint32_t* hdr, hipStream_t s) {
  const dim3 g(ew_grid(n)), b(EW_THREADS);
  switch (in_dtype) {
    case kE4M3: hipLaunchKernelGGL((amax_kernel<kE4M3>), g, b, 0, s, in, n, hdr); break;
    case kE5M2: hipLaunchKernelGGL((amax_kernel<kE5M2>), g, b, 0, s, in, n, hdr); break;
    case kF16: hipLaunchKernelGGL((amax_kernel<kF16>), g, b, 0, s, in, n, hdr); break;
    default: hipLaunchKernelGGL((amax_kernel<kF32>), g, b, 0, s, in, n, hdr); break;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------- rescale / cast / set_scaling

// Store the codes of a lane's 16 block elements (words w as encode16 packs
// them: FP8 4 codes per word, FP16 2) at their elements: the EPW codes of
// input word k go to element 64 k + lane (in units of EPW elements) of the
// block, as one store of EPW * (1 or 2) bytes.
template <int INF, int OUTF>
__device__ __forceinline__ void store_block(void* out, int64_t b, int lane, const uint32_t (&w)[8]) {
  constexpr int W = BlockLayout<INF>::W, EPW = BlockLayout<INF>::EPW;
  constexpr int OB = OUTF == kF16 ? 2 : 1;  // output bytes per element
  constexpr int WPW = EPW * OB / 4;         // packed 32-bit words per input word
  uint8_t* base = (uint8_t*)out + (b * 1024) * OB;
#pragma unroll
  for (int k = 0; k < W; ++k) {
    uint8_t* q = base + (int64_t)(64 * k + lane) * EPW * OB;
    if constexpr (WPW == 1) *(uint32_t*)q = w[k];
    else if constexpr (WPW == 2) *(uint2*)q = uint2{w[2 * k], w[2 * k + 1]};
    else if constexpr (WPW == 4) *(u4*)q = u4{w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]};
    else {
      *(u4*)q = u4{w[0], w[1], w[2], w[3]};
      *(u4*)(q + 16) = u4{w[4], w[5], w[6], w[7]};
    }
  }
}

template <int INF, int OUTF>
__global__ __launch_bounds__(EW_THREADS) void elementwise_kernel(ElemParams p) {
  using L = BlockLayout<INF>;
  int shift = 0, e_out = 0;
  if (p.rule != RULE_COPY) {
    const int e_in = p.hdr ? (int)p.hdr[1] : pow2_exponent(p.in_scale);
    if (p.rule == RULE_AMAX) e_out = clamp_e8m0(e_in + rescale_exponent(p.hdr[0], p.target));
    else if (p.rule == RULE_KEEP) e_out = e_in;
    else e_out = p.e_fixed;
    shift = e_out - e_in;
  }
  const bool sat = p.sat != 0;
  const bool fast = shift >= kFastShiftMinSub && shift <= kFastShiftMax;
  const float scale = fast ? pow2_float(shift) : 1.0f;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    if (p.rule == RULE_COPY) *p.out_scale = p.in_scale ? *p.in_scale : 1.0f;
    else *p.out_scale = pow2_float(e_out);
  }
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (EW_THREADS / 64) + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * (EW_THREADS / 64);
  const int64_t nb = p.n / 1024;
  auto cast_block = [&](const u4 (&w)[L::W], int64_t b) {
    uint32_t c[16];
    unpack_block<INF>(w, c);
#pragma unroll
    for (int i = 0; i < 16; ++i) c[i] = to_bits<INF>(c[i]);
    uint32_t o[8];
    encode16<OUTF>(c, shift, scale, fast, sat, o);
    store_block<INF, OUTF>(p.out, b, lane, o);
  };
  int64_t b = wave;
  for (; b + waves < nb; b += 2 * waves) {
    u4 w0[L::W], w1[L::W];
    load_block<INF>(p.in, b, lane, w0);
    load_block<INF>(p.in, b + waves, lane, w1);
    cast_block(w0, b);
    cast_block(w1, b + waves);
  }
  if (b < nb) {
    u4 w0[L::W];
    load_block<INF>(p.in, b, lane, w0);
    cast_block(w0, b);
  }
  if (blockIdx.x == 0)
    for (int64_t e = nb * 1024 + threadIdx.x; e < p.n; e += EW_THREADS)
      store1<OUTF>(p.out, e, cast_bits<OUTF>(to_bits<INF>(load1<INF>(p.in, e)), shift, sat));
}

template <int INF>
static void launch_elem_out(const ElemParams& p, int out_dtype, dim3 g, dim3 b, hipStream_t s) {
  if (out_dtype == kE4M3) hipLaunchKernelGGL((elementwise_kernel<INF, kE4M3>), g, b, 0, s, p);
  else if (out_dtype == kE5M2) hipLaunchKernelGGL((elementwise_kernel<INF, kE5M2>), g, b, 0, s, p);
  else hipLaunchKernelGGL((elementwise_kernel<INF, kF16>), g, b, 0, s, p);
}

hipError_t launch_elementwise(const ElemParams& p, int in_dtype, int out_dtype, hipStream_t s) {
  const dim3 g(ew_grid(p.n)), b(EW_THREADS);
  switch (in_dtype) {
    case kE4M3: launch_elem_out<kE4M3>(p, out_dtype, g, b, s); break;
    case kE5M2: launch_elem_out<kE5M2>(p, out_dtype, g, b, s); break;
    case kF16: launch_elem_out<kF16>(p, out_dtype, g, b, s); break;
    default: launch_elem_out<kF32>(p, out_dtype, g, b, s); break;
  }
  return hipGetLastError();
}

}  // namespace scalify
