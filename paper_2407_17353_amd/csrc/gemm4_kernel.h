// Persistent one-wave-per-SIMD scaled FP8 GEMM for gfx950: the FP8
// dot_general with fp32 accumulation of the scaled matmul (Section 3.2 /
// Algorithm 3; higher-precision accumulation of FP8 products, Appendix A)
// with its epilogue fused, and the single-pass form of the dynamic rescale
// (Section 3.3), whose statistic is the amax of the whole output.
//
// One workgroup of 4 waves per CU walks its share of the 256 x 256 output
// tiles (tile ids b, b + G, b + 2G, ... for workgroup b of a grid of G,
// mapped to tile origins by tile_origin), with the main loop of the 4-wave
// arrangement (WaveCfg<4>: each wave a 128 x 128 sub-tile whose 256
// accumulators stay in AGPRs named by AccTile, two barriers per k-step,
// loads two steps ahead, A fragments double-buffered by step parity). The
// k-steps of consecutive tiles form one stream: the loads issued during the
// last two steps of a tile are those of the next tile's first two steps, so
// they are in flight while the tile's epilogue runs. Every tile is given an
// even number of steps (a step past K loads zeros), so that a tile starts at
// even parity.
//
// Epilogues:
//   EPI_INTER16 / EPI_INTER32: every tile stores the pre-cast intermediate
//     (16-bit rounding-preserving encoding / fp32) for the cast kernel;
//   EPI_DIRECT: every tile stores its output codes, the shift known before
//     the GEMM (delayed rescale, or no rescale);
//   SP (single pass, with EPI_INTER16 / EPI_INTER32): every tile but the
//     workgroup's last stores the intermediate; the last one stays in the
//     accumulators. The workgroups then meet at a grid barrier on the amax
//     statistic (the barrier at the end of the kernel), derive the rescale exponent, cast the held
//     tile straight from the accumulators and cast their earlier tiles from
//     the intermediate.
#pragma once
#include "ew_util.h"
#include "gemm_kernel.h"

namespace scalify {

// LDS bytes per wave for staging the epilogue's stores.
constexpr int kStageWave = 4096;

// Header words of the single-pass barrier (zeroed by the matmul prologue).
constexpr int kHdrArrive = 5, kHdrState = 6, kHdrWritten = 7;
enum SpState : uint32_t { SP_RUNNING = 0, SP_COMPLETE = 1, SP_ABORTED = 2 };

// ---- casts without calls (usable while accumulators sit in AGPRs)

// 4 fp32 values times 2^-shift to FP8 format F, equal to cast_bits for every
// input: inside the fast window the conversion takes the power-of-two scale
// itself; outside it the values are first scaled by v_ldexp_f32, which is
// exact whenever the result is a normal fp32, while a result below 2^-126
// converts to a zero of its sign and an overflow to +-Inf, as the exact value
// would (the format's smallest subnormal is far above 2^-126, its largest
// value far below 2^128). NaN inputs give the NaN code with their sign.
template <int F>
__device__ __forceinline__ uint32_t cast4_fp8_any(const v4f& v, bool fast, float scale, int shift,
                                                  bool sat) {
  uint32_t u[4], x[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    u[i] = __float_as_uint(v[i]);
    x[i] = fast ? u[i] : __float_as_uint(__builtin_amdgcn_ldexpf(v[i], -shift));
  }
  uint32_t w = cast4_fp8_hw<F>(x[0], x[1], x[2], x[3], fast ? scale : 1.0f, sat);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t nanc = FmtTraits<F>::NANC | ((u[i] >> 24) & 0x80u);
    if (is_nan_bits(u[i])) w = (w & ~(0xFFu << (8 * i))) | (nanc << (8 * i));
  }
  return w;
}

// The same to FP16 (inv = 2^-shift inside the fast window), two codes per
// word.
__device__ __forceinline__ v2i cast4_f16_any(const v4f& v, bool fast, float inv, int shift,
                                            bool sat) {
  uint32_t u[4], x[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    u[i] = __float_as_uint(v[i]);
    x[i] = fast ? u[i] : __float_as_uint(__builtin_amdgcn_ldexpf(v[i], -shift));
  }
  const v2i h = cast4_f16_hw(x[0], x[1], x[2], x[3], fast ? inv : 1.0f, sat);
  uint32_t c[4] = {(uint32_t)h.x & 0xFFFFu, (uint32_t)h.x >> 16, (uint32_t)h.y & 0xFFFFu,
                   (uint32_t)h.y >> 16};
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (is_nan_bits(u[i])) c[i] = FmtTraits<kF16>::NANC | ((u[i] >> 16) & 0x8000u);
  return v2i{(int)(c[0] | (c[1] << 16)), (int)(c[2] | (c[3] << 16))};
}

// Running max of |a|, |b| and m (m >= 0), one instruction: the fast
// epilogues call it on values known not to be NaN.
__device__ __forceinline__ float max3_abs(float m, float a, float b) {
  float r;
  asm("v_max3_f32 %0, %1, |%2|, |%3|" : "=v"(r) : "v"(m), "v"(a), "v"(b));
  return r;
}

// 4 non-NaN fp32 values times inv = 2^-shift (inside the fast window) to
// FP16, two codes per word: the product is exact unless it leaves the fp32
// normal range (above it the conversion overflows as the exact value would,
// below it the value rounds to zero in FP16 either way; the product keeps
// the sign of a zero), converted with round to nearest even. SAT clamps the
// product to +-65504 first, which is what saturation gives for every value
// that would overflow.
template <bool SAT>
__device__ __forceinline__ v2i cvt4_f16_fast(float x0, float x1, float x2, float x3, float inv) {
  float y[4] = {x0 * inv, x1 * inv, x2 * inv, x3 * inv};
  if constexpr (SAT) {
#pragma unroll
    for (int i = 0; i < 4; ++i) y[i] = __builtin_amdgcn_fmed3f(y[i], -65504.0f, 65504.0f);
  }
  int lo, hi;
  asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(lo) : "v"(y[0]), "v"(y[1]));
  asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(hi) : "v"(y[2]), "v"(y[3]));
  return v2i{lo, hi};
}

// The cast kernel's arithmetic on one 16-element chunk of the intermediate
// (fp32 bits, or 16-bit encodings shifted into the top half), call-free.
template <int OUTF>
__device__ __forceinline__ void encode16_any(const uint32_t (&c)[16], bool fast, float scale,
                                             float inv, int shift, bool sat, uint32_t (&w)[8]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const v4f v = {__uint_as_float(c[4 * q]), __uint_as_float(c[4 * q + 1]),
                   __uint_as_float(c[4 * q + 2]), __uint_as_float(c[4 * q + 3])};
    if constexpr (OUTF == kF16) {
      const v2i h = cast4_f16_any(v, fast, inv, shift, sat);
      w[2 * q] = (uint32_t)h.x;
      w[2 * q + 1] = (uint32_t)h.y;
    } else {
      w[q] = cast4_fp8_any<OUTF>(v, fast, scale, shift, sat);
      w[4 + q] = 0u;
    }
  }
}

// Shift of the cast from the amax statistic (bits of max |acc|): the rescale
// exponent of Section 3.3 rounded down, e_out = clamp(e_w + e_c + e_r).
__device__ __forceinline__ int sp_shift(uint32_t amax_raw, int e_w, int e_c, int target,
                                        int* e_out_p) {
  int e_r = 0;
  if (amax_raw != 0u && amax_raw < 0x7F800000u) e_r = floor_log2_bits(amax_raw) - e_c - target;
  const int e_out = clamp_e8m0(e_w + e_c + e_r);
  *e_out_p = e_out;
  return e_out - e_w;
}

// OF: the output format the kernel casts to (EPI_DIRECT, SP), -1 for the
// intermediate-only kernels.
template <bool A_MN, bool B_KC, int FA, int FB, int EPI, bool MX, bool SP, int OF>
__global__ __launch_bounds__(256, 1) void gemm4_kernel(GemmParams p) {
  static_assert(!SP || EPI != EPI_DIRECT, "the single pass holds a tile of the intermediate kinds");
  static_assert((OF >= 0) == (SP || EPI == EPI_DIRECT), "an output format exactly when casting");
  static_assert(!SP || EPI == EPI_INTER32 || OF != kF16, "FP16 outputs take the fp32 intermediate");
  using C = WaveCfg<4>;
  constexpr int WAVES_N = C::WAVES_N, WTM = C::WTM, WTN = C::WTN;
  constexpr int MI = C::MI, NI = C::NI, BPW = C::BPW, LOADS_PER_STEP = C::LOADS_PER_STEP;
  __shared__ __attribute__((aligned(1024))) uint8_t sA0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sB0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sB1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sStage[4 * kStageWave];
  __shared__ float red[4];
  __shared__ uint32_t sp_word[2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = gridDim.x;
  const int T = p.tiles_m * p.tiles_n;
  const int ntiles = (T - (int)blockIdx.x + G - 1) / G;  // >= 1: G <= T

  const int M = p.M, N = p.N, K = p.K;
  const int KT = (K + BK - 1) / BK;
  const int KTe = KT < 2 ? 2 : KT + (KT & 1);  // steps per tile, even
  const int KT_full = K / BK;                 // k-steps entirely inside K
  const int krem = K - KT_full * BK;          // bytes of the partial last step (0 if none)
  const uint32_t lda = (uint32_t)p.lda, ldb = (uint32_t)p.ldb;
  const v4i ra = make_rsrc(p.a, p.a_bytes);
  const v4i rb = make_rsrc(p.b, p.b_bytes);

  // Per-load parts of the load offsets, per lane (load q of this wave's share
  // of a tile: block blk = wave * BPW + q): KC rows along M/N, MC rows along
  // K (see make_loader), so that a load adds one scalar to one register.
  // KC tiles also keep the k offset of the lane's 16-byte chunk per block
  // parity (loads at or past K go out of range).
  uint32_t qa[BPW], qb[BPW];
  int kca[2] = {0, 0}, kcb[2] = {0, 0};
  {
    const TileLoader la = make_loader<!A_MN, BPW>(lda, wave, lane);
    const TileLoader lb = make_loader<B_KC, BPW>(ldb, wave, lane);
#pragma unroll
    for (int q = 0; q < BPW; ++q) {
      const uint32_t blk = (uint32_t)(wave * BPW + q);
      qa[q] = blk * (A_MN ? 4u : 8u) * lda + la.lane_off[q & 1];
      qb[q] = blk * (B_KC ? 8u : 4u) * ldb + lb.lane_off[q & 1];
    }
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      kca[par] = la.kchunk[par];
      kcb[par] = lb.kchunk[par];
    }
  }

  // Load cursor: the (tile, k-step) whose loads are issued next, and the
  // scalar parts of its offsets (KC: row0 * ld + k0, MC: k0 * ld + row0).
  // Past the last tile the cursor stays at k-step KT, whose loads all fall
  // past K and read zeros without touching memory.
  int l_r = 0, l_kt = 0, l_m0, l_n0;
  uint32_t l_sa = 0, l_sb = 0;
  tile_origin(blockIdx.x, p.tiles_m, p.tiles_n, l_m0, l_n0);
  auto cursor_bases = [&]() {
    const uint32_t k0 = (uint32_t)(l_kt * BK);
    l_sa = A_MN ? k0 * lda + (uint32_t)l_m0 : (uint32_t)l_m0 * lda + k0;
    l_sb = B_KC ? (uint32_t)l_n0 * ldb + k0 : k0 * ldb + (uint32_t)l_n0;
  };
  cursor_bases();
  auto advance = [&]() {
    if (++l_kt >= KTe) {
      if (l_r + 1 < ntiles) {
        l_kt = 0;
        ++l_r;
        tile_origin(blockIdx.x + l_r * G, p.tiles_m, p.tiles_n, l_m0, l_n0);
      } else {
        l_kt = KT;
      }
    }
    cursor_bases();
  };
  // Load j of the cursor's step: j < BPW are A blocks, the rest B blocks.
  auto issue_one = [&](int j, uint8_t* dA, uint8_t* dB) {
    const int k0 = l_kt * BK;
    if (j < BPW) {
      uint32_t off = qa[j] + l_sa;
      if (!A_MN && k0 + kca[j & 1] >= K) off = (uint32_t)ra.z;
      load_lds16(ra, off, dA + (wave * BPW + j) * 1024);
    } else {
      const int q = j - BPW;
      uint32_t off = qb[q] + l_sb;
      if (B_KC && k0 + kcb[q & 1] >= K) off = (uint32_t)rb.z;
      load_lds16(rb, off, dB + (wave * BPW + q) * 1024);
    }
  };
  auto zero_tail = [&](uint8_t* dA, uint8_t* dB) {
    if (!A_MN) zero_tail_kc(dA, krem, tid);
    if (B_KC) zero_tail_kc(dB, krem, tid);
    __syncthreads();
  };

  // MX block scales, packed (see GemmParams): wave w stages group w of A
  // (half 0) and of B (half 1) of the cursor's step beside its tiles. Stage
  // layout: [2 k-step stages][A 1 KiB | B 1 KiB], tile group j at 256 j.
  uint8_t* sS = nullptr;
  if constexpr (MX) {
    __shared__ __attribute__((aligned(1024))) uint8_t s_mx[4096];
    sS = s_mx;
  }
  auto issue_scale_half = [&](int stage, bool is_b) {
    if constexpr (MX) {
      const int groups = is_b ? p.mx_groups_b : p.mx_groups_a;
      const int grp = (is_b ? l_n0 : l_m0) / 64 + wave;
      const v4i r = is_b ? make_rsrc(p.mx_b, p.mx_b_bytes) : make_rsrc(p.mx_a, p.mx_a_bytes);
      // (past the last tile l_kt = KT: past the array's k-steps, out of range)
      const uint32_t off = grp < groups
                               ? ((uint32_t)(l_kt * groups + grp) * 64u + (uint32_t)lane) * 4u
                               : (uint32_t)r.z;
      load_lds4(r, off, sS + stage * 2048 + (is_b ? 1024 : 0) + 256 * wave);
    }
  };
  auto scale_word = [&](int stage, int half, int j) -> int {
    return *(const int*)(sS + stage * 2048 + half * 1024 + 256 * j + 4 * lane);
  };

  const int wm = (wave / WAVES_N) * WTM;  // wave sub-tile
  const int wn = (wave % WAVES_N) * WTN;
  constexpr int DSA = A_MN ? 4 : 2;  // LDS reads per A fragment
  constexpr int DSB = B_KC ? 2 : 4;  // LDS reads per B fragment
  static_assert(LOADS_PER_STEP == 2 * MI, "two loads per row block");

  // Main loop schedule (per k-step kt of a tile; see the file comment of
  // gemm_kernel.h for the one-wave-per-SIMD arrangement):
  //   head(kt): column groups 0 .. H - 1, reading the B fragments of groups
  //     2 .. NI - 1 one LDS read per MFMA; barrier X after group 0 (every
  //     wave has read step kt's A fragments), then the A loads of the
  //     cursor's step (two ahead) into this step's A stage; barrier Y at the
  //     end (every wave has read step kt's B fragments and the next step has
  //     landed: only this head's A loads may still be in flight);
  //   tail(kt): groups H .. NI - 1, with the B loads of the cursor's step into
  //     this step's B stage and the reads of the next step's A fragments
  //     (other buffer) and B fragments 0, 1; then the cursor advances.
  constexpr int H = 6;
  static_assert(H >= 3 && H < NI && (NI - 2) * DSB <= H * MI, "head too short for its B reads");
  constexpr int TS = (NI - H) * MI;
  constexpr int AS = (H - 1) * MI;
  constexpr int BP = 2 * DSB;
  constexpr int RX = MI < (NI - 2) * DSB ? MI : (NI - 2) * DSB;
  v8i af[2][MI];
  v8i bf[NI];
  int sa[2][2] = {}, sb[2][2] = {};
  static_assert(!MX || (MI == 8 && NI == 8 && WTM == 128 && WTN == 128), "MX word layout");

  auto head = [&](auto par_tag, int kt) {
    constexpr int P = decltype(par_tag)::value;
    constexpr bool odd = P == 1;  // tiles have an even number of steps: kt & 1 == P
    uint8_t* cA = odd ? sA1 : sA0;
    uint8_t* cB = odd ? sB1 : sB0;
    static_for<0, H * MI>([&](auto I) {
      constexpr int i = decltype(I)::value;
      constexpr int ni = i / MI, mi = i % MI;
      if constexpr (MX)
        AccTile<mi * NI + ni>::template mfma_mx<FA, FB, ni & 3, mi & 3>(
            bf[ni], af[P][mi], sb[P][ni >> 2], sa[P][mi >> 2]);
      else
        AccTile<mi * NI + ni>::template mfma<FA, FB>(bf[ni], af[P][mi]);
      if constexpr (i < (NI - 2) * DSB) {
        constexpr int g = 2 + i / DSB;
        read_frag_part<B_KC, i % DSB, MX>(bf[g], cB, wn + 16 * g, lane);
      }
      if constexpr (i == MI - 1) {
        wait_lgkmcnt<RX>();
        __builtin_amdgcn_s_barrier();
      }
      if constexpr (i >= MI) {
        constexpr int j = i - MI;
        static_for<j * BPW / AS, (j + 1) * BPW / AS>([&](auto J) {
          issue_one(decltype(J)::value, cA, cB);
        });
        if constexpr (i + 1 == H * MI) issue_scale_half(odd, false);
      }
    });
    wait_vmcnt<BPW + (MX ? 1 : 0)>();
    wait_lgkmcnt<0>();
    __builtin_amdgcn_s_barrier();
    // the next step (the next tile's first one after the last step of a tile)
    const int nk = kt + 1 == KTe ? 0 : kt + 1;
    if (nk == KT_full && (krem & 15)) zero_tail(odd ? sA0 : sA1, odd ? sB0 : sB1);
  };
  auto tail = [&](auto par_tag, int kt) {
    constexpr int P = decltype(par_tag)::value;
    constexpr bool odd = P == 1;  // tiles have an even number of steps: kt & 1 == P
    uint8_t* cA = odd ? sA1 : sA0;
    uint8_t* cB = odd ? sB1 : sB0;
    uint8_t* nA = odd ? sA0 : sA1;
    uint8_t* nB = odd ? sB0 : sB1;
    static_for<0, TS>([&](auto I) {
      constexpr int i = decltype(I)::value;
      constexpr int mi = i / (NI - H), ni = H + i % (NI - H);
      if constexpr (MX)
        AccTile<mi * NI + ni>::template mfma_mx<FA, FB, ni & 3, mi & 3>(
            bf[ni], af[P][mi], sb[P][ni >> 2], sa[P][mi >> 2]);
      else
        AccTile<mi * NI + ni>::template mfma<FA, FB>(bf[ni], af[P][mi]);
      static_for<i * BPW / TS, (i + 1) * BPW / TS>([&](auto J) {
        issue_one(BPW + decltype(J)::value, cA, cB);
      });
      if constexpr (i + 1 == TS) issue_scale_half(odd, true);
      static_for<i * BP / TS, (i + 1) * BP / TS>([&](auto Q) {
        constexpr int q = decltype(Q)::value;
        read_frag_part<B_KC, q % DSB, MX>(bf[q / DSB], nB, wn + 16 * (q / DSB), lane);
      });
      static_for<i * (MI * DSA) / TS, (i + 1) * (MI * DSA) / TS>([&](auto Q) {
        constexpr int q = decltype(Q)::value;
        read_frag_part<!A_MN, q % DSA, MX>(af[P ^ 1][q / DSA], nA, wm + 16 * (q / DSA), lane);
      });
    });
    if constexpr (MX) {
      sa[P ^ 1][0] = scale_word(!odd, 0, wm / 64);
      sa[P ^ 1][1] = scale_word(!odd, 0, wm / 64 + 1);
      sb[P ^ 1][0] = scale_word(!odd, 1, wn / 64);
      sb[P ^ 1][1] = scale_word(!odd, 1, wn / 64 + 1);
    }
    advance();
  };

  // ---- epilogue helpers: lane holds C[m][n..n+3] of tile (mi, ni) at
  // m = m0 + wm + 16 mi + (lane & 15), n = n0 + wn + 16 ni + 4 (lane >> 4)
  const bool sat = p.sat != 0;
  const int e_w = (int)__builtin_amdgcn_readfirstlane(p.hdr[1]);
  // EPI_DIRECT: data' = acc * 2^-shift, shift from the prologue
  const int d_shift = EPI == EPI_DIRECT ? (int)__builtin_amdgcn_readfirstlane(p.hdr[2]) : 0;
  // Block-scaled accumulators may be fp32 subnormals (the plain ones never are).
  auto fast_of = [&](int sh) { return sh >= (MX ? kFastShiftMinSub : -kFastShiftMax) && sh <= kFastShiftMax; };

  // Stores of a wave tile inside the matrix, staged through the wave's own
  // 4 KiB of LDS so that each store writes 16 bytes per lane and whole rows
  // of the wave tile (a 16-row block of ESZ = 2 byte elements, or a 32-row
  // block of 1 byte codes, per round). group(t) gives the packed elements
  // of accumulator tile t (4 of them: 4 ESZ bytes) and folds the statistic;
  // a lane writes them at its row and column, the 16-byte chunks of a row
  // permuted by the row (XOR) so that the writes and the row reads spread
  // over the LDS banks. LDS instructions of one wave complete in order, so
  // a round's writes reuse the region after the previous round's reads.
  auto staged = [&](auto esz_tag, uint8_t* base, int64_t ld, int m0, int n0, auto&& group) {
    constexpr int ESZ = decltype(esz_tag)::value;
    constexpr int RB = 128 * ESZ;    // bytes of a wave-tile row
    constexpr int CPR = RB / 16;     // 16-byte chunks per row
    constexpr int MPR = 2 / ESZ;     // accumulator-tile rows (of 16) per round
    constexpr int LPR = 64 / CPR;    // rows per read
    uint8_t* st = sStage + wave * kStageWave;
    const int r = lane & 15, q = lane >> 4;
    static_for<0, MI / MPR>([&](auto RD) {
      constexpr int rd = decltype(RD)::value;
      static_for<0, MPR * NI>([&](auto I) {
        constexpr int i = decltype(I)::value;
        constexpr int mi = rd * MPR + i / NI, ni = i % NI;
        const int rr = 16 * (mi % MPR) + r;
        const int chunk = ESZ == 2 ? 2 * ni + (q >> 1) : ni;
        const int off = ESZ == 2 ? 8 * (q & 1) : 4 * q;
        uint8_t* a = st + rr * RB + 16 * (chunk ^ (rr & (CPR - 1))) + off;
        const auto w = group(std::integral_constant<int, mi * NI + ni>{});
        if constexpr (ESZ == 2)
          *(v2i*)a = w;
        else
          *(uint32_t*)a = w;
      });
      wait_lgkmcnt<0>();
      u4 d[4];
      static_for<0, 4>([&](auto J) {
        constexpr int j = decltype(J)::value;
        const int R = j * LPR + lane / CPR, cc = lane % CPR;
        d[j] = *(const u4*)(st + R * RB + 16 * (cc ^ (R & (CPR - 1))));
      });
      wait_lgkmcnt<0>();
      static_for<0, 4>([&](auto J) {
        constexpr int j = decltype(J)::value;
        const int R = j * LPR + lane / CPR, cc = lane % CPR;
        const int64_t row = m0 + wm + 16 * rd * MPR + R;
        *(u4*)(base + (row * ld + n0 + wn + cc * (16 / ESZ)) * ESZ) = d[j];
      });
    });
  };

  // Store the tile at (m0, n0) from the accumulators: OUTF < 0 the
  // intermediate of EPI, else output codes of format OUTF with `shift`;
  // fold |acc| of the valid elements into lmax; ZERO: clear the
  // accumulators for the next tile; acc_out exports the raw accumulators.
  auto store_tile = [&](auto outf_tag, auto zero_tag, int m0, int n0, int shift, float& lmax) {
    constexpr int OUTF = decltype(outf_tag)::value;
    constexpr bool ZERO = decltype(zero_tag)::value;
    const bool fast = fast_of(shift);
    const float scale = fast ? pow2_float(shift) : 1.0f;
    const float inv = fast ? pow2_float(-shift) : 1.0f;
    const int mb = m0 + wm + (lane & 15);
    const int nb = n0 + wn + 4 * (lane >> 4);
    // one 4-value group: codes or intermediate at row m, column n (cols valid)
    auto put = [&](const v4f& v, int m, int n, int cols) {
      if constexpr (OUTF == kF16) {
        const v2i w = cast4_f16_any(v, fast, inv, shift, sat);
        uint16_t* q = (uint16_t*)p.out + (int64_t)m * p.ldc + n;
        if (cols >= 4) {
          *(v2i*)q = w;
        } else {
          q[0] = (uint16_t)w.x;
          if (cols > 1) q[1] = (uint16_t)((uint32_t)w.x >> 16);
          if (cols > 2) q[2] = (uint16_t)w.y;
        }
      } else if constexpr (OUTF >= 0) {
        const uint32_t w = cast4_fp8_any<OUTF>(v, fast, scale, shift, sat);
        uint8_t* q = (uint8_t*)p.out + (int64_t)m * p.ldc + n;
        if (cols >= 4) {
          *(uint32_t*)q = w;
        } else {
          q[0] = (uint8_t)w;
          if (cols > 1) q[1] = (uint8_t)(w >> 8);
          if (cols > 2) q[2] = (uint8_t)(w >> 16);
        }
      } else if constexpr (EPI == EPI_INTER16) {
        // bits 16.. of u | ((u & 0xFFFF) + 0xFFFF) are sticky16(u): the
        // added term sets bit 16 exactly when a lower bit is set
        uint32_t x[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t u = __float_as_uint(v[k]);
          x[k] = u | ((u & 0xFFFFu) + 0xFFFFu);
        }
        *(v2i*)((uint16_t*)p.inter + (int64_t)m * p.ldw + n) =
            v2i{(int)__builtin_amdgcn_perm(x[1], x[0], 0x07060302u),
                (int)__builtin_amdgcn_perm(x[3], x[2], 0x07060302u)};
      } else {
        *(v4f*)((float*)p.inter + (int64_t)m * p.ldw + n) = v;  // (ldw: 16 elements)
      }
    };
    const bool inside = !p.acc_out && m0 + wm + 16 * MI <= M && n0 + wn + 16 * NI <= N;
    // the staged stores write 16 aligned bytes per lane
    const bool stage_ok = OUTF < 0 ? (p.ldw & 7) == 0 && ((uintptr_t)p.inter & 15) == 0
                                   : ((p.ldc * (OUTF == kF16 ? 2 : 1)) & 15) == 0 &&
                                         ((uintptr_t)p.out & 15) == 0;
    if constexpr (OUTF >= 0) {
      // Codes of a wave tile inside the matrix with the shift inside the fast
      // window: the conversion scales by itself, saturation is chosen once
      // for the tile, and a group holding a NaN (rare) takes a branch that
      // puts the NaN codes in and keeps the NaN out of the statistic.
      auto codes = [&](auto sat_tag) {
        constexpr bool SAT = decltype(sat_tag)::value;
        constexpr int ESZ = OUTF == kF16 ? 2 : 1;
        staged(std::integral_constant<int, ESZ>{}, (uint8_t*)p.out, p.ldc, m0, n0, [&](auto I) {
          constexpr int t = decltype(I)::value;
          const v4f v = AccTile<t>::read();
          if constexpr (ZERO) AccTile<t>::zero();
          float x[4] = {v[0], v[1], v[2], v[3]};
          if constexpr (OUTF == kF16) {
            v2i w = cvt4_f16_fast<SAT>(x[0], x[1], x[2], x[3], inv);
            if (__builtin_expect(x[0] != x[0] || x[1] != x[1] || x[2] != x[2] || x[3] != x[3], 0)) {
              uint32_t h[4] = {(uint32_t)w.x & 0xFFFFu, (uint32_t)w.x >> 16, (uint32_t)w.y & 0xFFFFu,
                               (uint32_t)w.y >> 16};
#pragma unroll
              for (int i = 0; i < 4; ++i)
                if (x[i] != x[i]) {
                  h[i] = FmtTraits<kF16>::NANC | ((__float_as_uint(x[i]) >> 16) & 0x8000u);
                  x[i] = 0.f;
                }
              w = v2i{(int)(h[0] | (h[1] << 16)), (int)(h[2] | (h[3] << 16))};
            }
            lmax = max3_abs(max3_abs(lmax, x[0], x[1]), x[2], x[3]);
            return w;
          } else {
            uint32_t w = cast4_fp8_hw<OUTF>(__float_as_uint(x[0]), __float_as_uint(x[1]),
                                            __float_as_uint(x[2]), __float_as_uint(x[3]), scale, SAT);
            if (__builtin_expect(x[0] != x[0] || x[1] != x[1] || x[2] != x[2] || x[3] != x[3], 0)) {
#pragma unroll
              for (int i = 0; i < 4; ++i)
                if (x[i] != x[i]) {
                  const uint32_t c = FmtTraits<OUTF>::NANC | ((__float_as_uint(x[i]) >> 24) & 0x80u);
                  w = (w & ~(0xFFu << (8 * i))) | (c << (8 * i));
                  x[i] = 0.f;
                }
            }
            lmax = max3_abs(max3_abs(lmax, x[0], x[1]), x[2], x[3]);
            return w;
          }
        });
      };
      if (inside && fast && stage_ok) {
        if (sat)
          codes(std::true_type{});
        else
          codes(std::false_type{});
        return;
      }
    }
    if constexpr (OUTF < 0 && EPI == EPI_INTER16) {
      if (inside && stage_ok) {
        staged(std::integral_constant<int, 2>{}, (uint8_t*)p.inter, p.ldw, m0, n0, [&](auto I) {
          constexpr int t = decltype(I)::value;
          const v4f v = AccTile<t>::read();
          if constexpr (ZERO) AccTile<t>::zero();
          lmax = fmaxf(lmax, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
          uint32_t x[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const uint32_t u = __float_as_uint(v[k]);
            x[k] = u | ((u & 0xFFFFu) + 0xFFFFu);  // sticky16(u) in bits 16..
          }
          return v2i{(int)__builtin_amdgcn_perm(x[1], x[0], 0x07060302u),
                     (int)__builtin_amdgcn_perm(x[3], x[2], 0x07060302u)};
        });
        return;
      }
    }
    if (inside) {
      // wave tile inside the matrix: no per-element checks
      static_for<0, MI * NI>([&](auto I) {
        constexpr int t = decltype(I)::value;
        constexpr int mi = t / NI, ni = t % NI;
        const v4f v = AccTile<t>::read();
        if constexpr (ZERO) AccTile<t>::zero();
        lmax = fmaxf(lmax, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
        put(v, mb + 16 * mi, nb + 16 * ni, 4);
      });
    } else {
      static_for<0, MI * NI>([&](auto I) {
        constexpr int t = decltype(I)::value;
        constexpr int mi = t / NI, ni = t % NI;
        const v4f v = AccTile<t>::read();
        if constexpr (ZERO) AccTile<t>::zero();
        const int m = mb + 16 * mi;
        const int n = nb + 16 * ni;
        if (m < M && n < N) {
          const int cols = min(N - n, 4);
          lmax = fmaxf(lmax, fabsf(v[0]));
          if (cols > 1) lmax = fmaxf(lmax, fabsf(v[1]));
          if (cols > 2) lmax = fmaxf(lmax, fabsf(v[2]));
          if (cols > 3) lmax = fmaxf(lmax, fabsf(v[3]));
          put(v, m, n, cols);
          if (p.acc_out) {
            float* q = p.acc_out + (int64_t)m * N + n;
            q[0] = v[0];
            if (cols > 1) q[1] = v[1];
            if (cols > 2) q[2] = v[2];
            if (cols > 3) q[3] = v[3];
          }
        }
      });
    }
  };
  using OI = std::integral_constant<int, -1>;
  // Output codes of the tile (format OF).
  auto store_codes = [&](auto zero_tag, int m0, int n0, int shift, float& lmax) {
    store_tile(std::integral_constant<int, OF>{}, zero_tag, m0, n0, shift, lmax);
  };

  // ---- prologue: the first two steps of the first tile
#pragma unroll
  for (int j = 0; j < LOADS_PER_STEP; ++j) issue_one(j, sA0, sB0);
  issue_scale_half(0, false);
  issue_scale_half(0, true);
  advance();
#pragma unroll
  for (int j = 0; j < LOADS_PER_STEP; ++j) issue_one(j, sA1, sB1);
  issue_scale_half(1, false);
  issue_scale_half(1, true);
  advance();
  static_for<0, MI * NI>([&](auto I) { AccTile<decltype(I)::value>::zero(); });
  wait_vmcnt<LOADS_PER_STEP + (MX ? 2 : 0)>();
  __syncthreads();
  if (KT_full == 0 && (krem & 15)) zero_tail(sA0, sB0);
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) af[0][mi] = read_frag<!A_MN, MX>(sA0, wm + 16 * mi, lane);
  bf[0] = read_frag<B_KC, MX>(sB0, wn, lane);
  bf[1] = read_frag<B_KC, MX>(sB0, wn + 16, lane);
  if constexpr (MX) {
    sa[0][0] = scale_word(0, 0, wm / 64);
    sa[0][1] = scale_word(0, 0, wm / 64 + 1);
    sb[0][0] = scale_word(0, 1, wn / 64);
    sb[0][1] = scale_word(0, 1, wn / 64 + 1);
  }
  mfma_drain();

  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  int c_r = 0, c_m0, c_n0;  // the tile being computed
  tile_origin(blockIdx.x, p.tiles_m, p.tiles_n, c_m0, c_n0);
  float lmax = 0.f;
  head(P0{}, 0);
  for (int kt = 0;;) {
    tail(P0{}, kt);
    head(P1{}, kt + 1);
    tail(P1{}, kt + 1);
    kt += 2;
    if (kt == KTe) {
      kt = 0;
      const bool last = c_r + 1 == ntiles;
      if (SP && last) break;  // held in the accumulators
      mfma_drain();
      if constexpr (EPI == EPI_DIRECT)
        store_codes(std::true_type{}, c_m0, c_n0, d_shift, lmax);
      else
        store_tile(OI{}, std::true_type{}, c_m0, c_n0, 0, lmax);
      if (last) break;
      ++c_r;
      tile_origin(blockIdx.x + c_r * G, p.tiles_m, p.tiles_n, c_m0, c_n0);
      mfma_drain();  // the zeroing writes before the next MFMAs read them
    }
    head(P0{}, kt);
  }
  wait_vmcnt<0>();  // the out-of-range loads past the last tile

  if constexpr (SP) {
    // max |acc| of the held tile's valid elements, then the workgroup's
    // statistic (its accumulators are exported, when asked, by the cast)
    mfma_drain();
    const int mb = c_m0 + wm + (lane & 15);
    const int nb = c_n0 + wn + 4 * (lane >> 4);
    const bool inside = c_m0 + wm + 16 * MI <= M && c_n0 + wn + 16 * NI <= N;
    // (the uniform test outside the loops, and per-lane selects inside, keep
    // each loop straight-line: a tile's values are folded before the next
    // tile is read, instead of all 256 accumulators being held at once)
    if (inside) {
      static_for<0, MI * NI>([&](auto I) {
        const v4f v = AccTile<decltype(I)::value>::read();
        lmax = fmaxf(lmax, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
        __builtin_amdgcn_sched_barrier(0);
      });
    } else {
      static_for<0, MI * NI>([&](auto I) {
        constexpr int t = decltype(I)::value;
        constexpr int mi = t / NI, ni = t % NI;
        const v4f v = AccTile<t>::read();
        const int m = mb + 16 * mi, n = nb + 16 * ni;
        const int cols = m < M ? max(0, min(N - n, 4)) : 0;  // valid columns of the group
        const float a0 = cols > 0 ? fabsf(v[0]) : 0.f, a1 = cols > 1 ? fabsf(v[1]) : 0.f;
        const float a2 = cols > 2 ? fabsf(v[2]) : 0.f, a3 = cols > 3 ? fabsf(v[3]) : 0.f;
        lmax = fmaxf(lmax, fmaxf(fmaxf(a0, a1), fmaxf(a2, a3)));
        __builtin_amdgcn_sched_barrier(0);
      });
    }
  }
  // amax of |acc| over the valid elements (fmaxf ignores NaN): wave
  // butterfly, then across the waves, then one atomic max per workgroup on
  // the fp32 bits (non-negative floats order like their bits).
  for (int off = 32; off > 0; off >>= 1) lmax = fmaxf(lmax, __shfl_xor(lmax, off, 64));
  if (lane == 0) red[wave] = lmax;
  __syncthreads();
  if constexpr (!SP) {
    if (tid == 0) {
      const float wmax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
      atomicMax(p.hdr, __float_as_uint(wmax));
    }
    return;
  } else {
    // Grid barrier on the statistic. Thread 0 adds the workgroup's max
    // (atomic, performed before the arrival is counted), counts its arrival
    // and waits for the state word: the last arrival sets it
    // COMPLETE. The wait is bounded (p.spin_ticks of the 100 MHz real-time
    // counter, polled every few hundred cycles): a workgroup that
    // runs out sets ABORTED unless the state has changed; whichever of the
    // two is set first decides for every workgroup. COMPLETE: every
    // statistic is in, each workgroup casts its own tiles. ABORTED (the grid
    // was not co-resident): each workgroup writes its held tile to the
    // intermediate too, and the last one to have done so casts every tile.
    //
    // Tiles cast from the intermediate (this workgroup's earlier ones, or
    // every tile after an abort) are streamed in batches: per tile a thread
    // takes the 16-column chunk tid & 15 of rows (tid >> 4) + 16 j, j < 16,
    // CH chunks per batch held as raw 16-byte words; right after a chunk is
    // cast and stored, the load of the same slot one batch ahead is issued,
    // so CH chunks per thread (64 KiB per CU) stay in flight. The first
    // batch of the workgroup's own tiles is loaded after the arrival, before
    // the barrier wait (its own stores, visible to the workgroup after the
    // barrier above).
    constexpr int U = EPI == EPI_INTER32 ? 4 : 2;   // 16-byte words per chunk
    constexpr int CH = EPI == EPI_INTER32 ? 4 : 8;   // chunks per batch (64 VGPRs)
    constexpr int BPT = 16 / CH;                     // batches per tile
    constexpr int ESZ = EPI == EPI_INTER32 ? 4 : 2;  // bytes per intermediate element
    constexpr int SF = OF == kF16 ? kF16 : kE4M3;    // output storage: 2 or 1 byte
    u4 raw[CH][U];
    auto tile_of = [&](bool all, int r, int& m0, int& n0) {
      tile_origin(all ? r : (int)blockIdx.x + r * G, p.tiles_m, p.tiles_n, m0, n0);
    };
    auto load_slot = [&](auto I, int m0, int n0, int sub) {
      constexpr int i = decltype(I)::value;
      const int m = m0 + (tid >> 4) + 16 * (sub * CH + i);
      const int n = n0 + 16 * (tid & 15);
      if (m < M && n < N) {
        const u4* q = (const u4*)((const uint8_t*)p.inter + ((int64_t)m * p.ldw + n) * ESZ);
#pragma unroll
        for (int h = 0; h < U; ++h) raw[i][h] = q[h];
      }
    };
    // MODE 0: any shift (encode16_any); 1 / 2: the shift inside the fast
    // window, saturating / not (the conversion scales by itself; a group
    // holding a NaN takes a branch that puts the NaN codes in)
    auto cast_slot = [&](auto I, auto mode_tag, int m0, int n0, int sub, int shift, bool fast,
                         float scale, float inv) {
      constexpr int i = decltype(I)::value;
      constexpr int MODE = decltype(mode_tag)::value;
      const int m = m0 + (tid >> 4) + 16 * (sub * CH + i);
      const int n = n0 + 16 * (tid & 15);
      if (m < M && n < N) {
        uint32_t c[16];
#pragma unroll
        for (int h = 0; h < U; ++h)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            if constexpr (EPI == EPI_INTER32) {
              c[4 * h + k] = raw[i][h][k];
            } else {  // 16-bit encodings into the top half of an fp32
              c[8 * h + 2 * k] = raw[i][h][k] << 16;
              c[8 * h + 2 * k + 1] = raw[i][h][k] & 0xFFFF0000u;
            }
          }
        uint32_t w[8];
        if constexpr (MODE == 0) {
          encode16_any<(OF < 0 ? kE4M3 : OF)>(c, fast, scale, inv, shift, sat, w);
        } else {
          constexpr bool SAT = MODE == 1;
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const uint32_t* u = c + 4 * g;
            const bool nan = is_nan_bits(u[0]) || is_nan_bits(u[1]) || is_nan_bits(u[2]) ||
                             is_nan_bits(u[3]);
            if constexpr (OF == kF16) {
              v2i h = cvt4_f16_fast<SAT>(__uint_as_float(u[0]), __uint_as_float(u[1]),
                                         __uint_as_float(u[2]), __uint_as_float(u[3]), inv);
              if (__builtin_expect(nan, 0)) {
                uint32_t hh[4] = {(uint32_t)h.x & 0xFFFFu, (uint32_t)h.x >> 16,
                                  (uint32_t)h.y & 0xFFFFu, (uint32_t)h.y >> 16};
#pragma unroll
                for (int k = 0; k < 4; ++k)
                  if (is_nan_bits(u[k])) hh[k] = FmtTraits<kF16>::NANC | ((u[k] >> 16) & 0x8000u);
                h = v2i{(int)(hh[0] | (hh[1] << 16)), (int)(hh[2] | (hh[3] << 16))};
              }
              w[2 * g] = (uint32_t)h.x;
              w[2 * g + 1] = (uint32_t)h.y;
            } else {
              constexpr int F = OF < 0 ? kE4M3 : OF;
              uint32_t x = cast4_fp8_hw<F>(u[0], u[1], u[2], u[3], scale, SAT);
              if (__builtin_expect(nan, 0)) {
#pragma unroll
                for (int k = 0; k < 4; ++k)
                  if (is_nan_bits(u[k])) {
                    const uint32_t nc = FmtTraits<F>::NANC | ((u[k] >> 24) & 0x80u);
                    x = (x & ~(0xFFu << (8 * k))) | (nc << (8 * k));
                  }
              }
              w[g] = x;
              w[4 + g] = 0u;
            }
          }
        }
        const int64_t e = (int64_t)m * p.ldc + n;
        if (n + 16 <= N) {
          store_words16<SF>(p.out, e, w);
        } else {
          for (int k = 0; k < N - n; ++k) store1<SF>(p.out, e + k, word_code<SF>(w, k));
        }
      }
    };
    // Cast `count` tiles of the list (all: every tile, else this workgroup's
    // earlier ones); `loaded`: the first batch is already in flight.
    auto cast_tiles = [&](bool all, int count, bool loaded, int shift) {
      const bool fast = fast_of(shift);
      const float scale = fast ? pow2_float(shift) : 1.0f;
      const float inv = fast ? pow2_float(-shift) : 1.0f;
      const int nb = count * BPT;
      if (nb == 0) return;
      int cm0, cn0;  // origin of the batch being cast
      tile_of(all, 0, cm0, cn0);
      if (!loaded) static_for<0, CH>([&](auto I) { load_slot(I, cm0, cn0, 0); });
      auto batches = [&](auto mode_tag) {
        for (int bi = 0; bi < nb; ++bi) {
          const int sub = bi % BPT, nbi = bi + 1, nsub = nbi % BPT;
          int nm0 = cm0, nn0 = cn0;  // origin of the next batch
          if (nbi < nb && nsub == 0) tile_of(all, nbi / BPT, nm0, nn0);
          static_for<0, CH>([&](auto I) {
            cast_slot(I, mode_tag, cm0, cn0, sub, shift, fast, scale, inv);
            if (nbi < nb) load_slot(I, nm0, nn0, nsub);
          });
          cm0 = nm0;
          cn0 = nn0;
        }
      };
      if (!fast)
        batches(std::integral_constant<int, 0>{});
      else if (sat)
        batches(std::integral_constant<int, 1>{});
      else
        batches(std::integral_constant<int, 2>{});
    };
    const bool own = ntiles > 1;
    if (tid == 0) {
      const float wmax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
      __hip_atomic_fetch_max(p.hdr, __float_as_uint(wmax), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // the max is performed before the arrival is counted (nothing else of
      // this workgroup needs to be visible to the others unless the barrier
      // aborts, which releases its stores itself)
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      const uint32_t arrived = __hip_atomic_fetch_add(p.hdr + kHdrArrive, 1u, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT) + 1u;
      if (arrived == (uint32_t)G) {
        uint32_t e = SP_RUNNING;
        __hip_atomic_compare_exchange_strong(p.hdr + kHdrState, &e, (uint32_t)SP_COMPLETE,
                                             __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    // the first batch of the earlier tiles in flight during the wait (issued
    // after the arrival, which waits for every load of its wave)
    if (own) {
      int m0, n0;
      tile_of(false, 0, m0, n0);
      static_for<0, CH>([&](auto I) { load_slot(I, m0, n0, 0); });
    }
    if (tid == 0) {
      uint32_t st = __hip_atomic_load(p.hdr + kHdrState, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // (a poll takes at least the sleep, 640 cycles or 30 ticks: the poll
      // count bounds the wait even if the counter did not advance)
      const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
      const int64_t max_polls = p.spin_ticks / 8 + 64;
      for (int64_t it = 0; st == SP_RUNNING && it < max_polls &&
                           (int64_t)(__builtin_amdgcn_s_memrealtime() - t0) < p.spin_ticks;
           ++it) {
        __builtin_amdgcn_s_sleep(10);
        st = __hip_atomic_load(p.hdr + kHdrState, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      if (st == SP_RUNNING) {
        uint32_t e = SP_RUNNING;
        __hip_atomic_compare_exchange_strong(p.hdr + kHdrState, &e, (uint32_t)SP_ABORTED,
                                             __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        st = __hip_atomic_load(p.hdr + kHdrState, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      sp_word[0] = st;
      sp_word[1] = __hip_atomic_load(p.hdr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    const uint32_t st = sp_word[0];
    bool cast_all = false;
    if (st == SP_ABORTED) {
      // the held tile joins the intermediate; the last writer casts everything
      float unused = 0.f;
      store_tile(OI{}, std::false_type{}, c_m0, c_n0, 0, unused);
      // every thread's intermediate stores (all tiles of this workgroup)
      // device-wide before the count; the last writer acquires them all
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      __syncthreads();
      if (tid == 0) {
        const uint32_t w = __hip_atomic_fetch_add(p.hdr + kHdrWritten, 1u, __ATOMIC_ACQ_REL,
                                                  __HIP_MEMORY_SCOPE_AGENT) + 1u;
        sp_word[0] = w == (uint32_t)G ? 1u : 0u;
        sp_word[1] = __hip_atomic_load(p.hdr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __syncthreads();
      if (!sp_word[0]) return;
      cast_all = true;
    }
    const uint32_t amax_raw = sp_word[1];
    int e_out;
    const int shift = sp_shift(amax_raw, e_w, p.e_c, p.target, &e_out);
    if (tid == 0 && (blockIdx.x == 0 || cast_all)) {
      *p.out_scale = pow2_float(e_out);
      if (p.amax_out) *p.amax_out = __uint_as_float(amax_raw) * pow2_float(-p.e_c);
    }
    if (!cast_all) {
      float unused = 0.f;
      store_codes(std::false_type{}, c_m0, c_n0, shift, unused);
      cast_tiles(false, ntiles - 1, true, shift);
    } else {
      cast_tiles(true, T, false, shift);
    }
  }
}

// ---- launches. Families, each instantiated in a source file of its own so
// that they compile in parallel:
//   launch_layout<A_MN, B_KC, false> (gemm_<layout>.hip): the 4-wave kernel
//     with the intermediate (GEMM + cast kernel);
//   launch_layout_direct<A_MN, B_KC> (gemm_<layout>_direct.hip): the 4-wave
//     kernel with the direct cast (delayed or no rescale);
//   launch_layout_sp<A_MN, B_KC> (gemm_<layout>_sp.hip): the single pass;
//   launch_layout<A_MN, B_KC, true> (gemm_<layout>_fused.hip): the 8-wave
//     kernel with the fused residual add / activation / channel scales;
//   launch_layout_mx<A_MN, B_KC> (gemm_<layout>_mx.hip, direct cast or the
//   fp32 intermediate) and launch_layout_mx_sp<A_MN, B_KC>
//   (gemm_<layout>_mx_sp.hip, single pass): MX block scales.
template <bool A_MN, bool B_KC, bool FUSE>
hipError_t launch_layout(const GemmParams& p, int fa, int fb, int epi, hipStream_t s);
template <bool A_MN, bool B_KC>
hipError_t launch_layout_direct(const GemmParams& p, int fa, int fb, int epi, hipStream_t s);
template <bool A_MN, bool B_KC>
hipError_t launch_layout_sp(const GemmParams& p, int fa, int fb, int epi, hipStream_t s);
template <bool A_MN, bool B_KC>
hipError_t launch_layout_mx(const GemmParams& p, int fa, int fb, int epi, hipStream_t s);
template <bool A_MN, bool B_KC>
hipError_t launch_layout_mx_sp(const GemmParams& p, int fa, int fb, int epi, hipStream_t s);

// The persistent kernel runs p.grid workgroups (host: gemm4_grid).
template <bool A_MN, bool B_KC, int FA, int FB, int EPI, bool MX, bool SP, int OF>
hipError_t launch4(const GemmParams& p, hipStream_t s) {
  hipLaunchKernelGGL((gemm4_kernel<A_MN, B_KC, FA, FB, EPI, MX, SP, OF>), dim3(p.grid), dim3(256),
                     0, s, p);
  return hipGetLastError();
}

// The 8-wave kernel: one workgroup per tile.
template <bool A_MN, bool B_KC, int FA, int FB, int EPI, bool FUSE, bool CH, bool MX>
hipError_t launch8(const GemmParams& p, hipStream_t s) {
  hipLaunchKernelGGL((gemm_kernel<A_MN, B_KC, FA, FB, EPI, FUSE, 8, CH, MX>),
                     dim3(p.tiles_m * p.tiles_n), dim3(WaveCfg<8>::NTHR), 0, s, p);
  return hipGetLastError();
}

// Dispatch over the format pair of A and B: F<FA, FB>::run(p, s).
template <template <int, int> class F>
hipError_t by_formats(const GemmParams& p, int fa, int fb, hipStream_t s) {
  if (fa == kE4M3 && fb == kE4M3) return F<kE4M3, kE4M3>::run(p, s);
  if (fa == kE4M3 && fb == kE5M2) return F<kE4M3, kE5M2>::run(p, s);
  if (fa == kE5M2 && fb == kE4M3) return F<kE5M2, kE4M3>::run(p, s);
  return F<kE5M2, kE5M2>::run(p, s);
}

template <bool A_MN, bool B_KC, bool FUSE>
struct PlainFamily {
  template <int FA, int FB>
  struct F {
    static hipError_t run(const GemmParams& p, hipStream_t s) {
      if constexpr (FUSE) {
        const bool ch = p.ch_a || p.ch_b;
        if (p.epi == EPI_DIRECT)
          return ch ? launch8<A_MN, B_KC, FA, FB, EPI_DIRECT, true, true, false>(p, s)
                    : launch8<A_MN, B_KC, FA, FB, EPI_DIRECT, true, false, false>(p, s);
        return ch ? launch8<A_MN, B_KC, FA, FB, EPI_INTER32, true, true, false>(p, s)
                  : launch8<A_MN, B_KC, FA, FB, EPI_INTER32, true, false, false>(p, s);
      } else {
        if (p.epi == EPI_INTER16) return launch4<A_MN, B_KC, FA, FB, EPI_INTER16, false, false, -1>(p, s);
        return launch4<A_MN, B_KC, FA, FB, EPI_INTER32, false, false, -1>(p, s);
      }
    }
  };
};

template <bool A_MN, bool B_KC, bool MX>
struct DirectFamily {
  template <int FA, int FB>
  struct F {
    static hipError_t run(const GemmParams& p, hipStream_t s) {
      // (block scales: the fp32 intermediate for the cast kernel also here)
      if (MX && p.epi == EPI_INTER32) return launch4<A_MN, B_KC, FA, FB, EPI_INTER32, MX, false, -1>(p, s);
      if (p.out_fmt == kE4M3) return launch4<A_MN, B_KC, FA, FB, EPI_DIRECT, MX, false, kE4M3>(p, s);
      if (p.out_fmt == kE5M2) return launch4<A_MN, B_KC, FA, FB, EPI_DIRECT, MX, false, kE5M2>(p, s);
      return launch4<A_MN, B_KC, FA, FB, EPI_DIRECT, MX, false, kF16>(p, s);
    }
  };
};

template <bool A_MN, bool B_KC, bool MX>
struct SpFamily {
  template <int FA, int FB>
  struct F {
    static hipError_t run(const GemmParams& p, hipStream_t s) {
      if constexpr (MX) {
        if (p.out_fmt == kE4M3) return launch4<A_MN, B_KC, FA, FB, EPI_INTER32, true, true, kE4M3>(p, s);
        if (p.out_fmt == kE5M2) return launch4<A_MN, B_KC, FA, FB, EPI_INTER32, true, true, kE5M2>(p, s);
        return launch4<A_MN, B_KC, FA, FB, EPI_INTER32, true, true, kF16>(p, s);
      } else {
        if (p.out_fmt == kE4M3) return launch4<A_MN, B_KC, FA, FB, EPI_INTER16, false, true, kE4M3>(p, s);
        if (p.out_fmt == kE5M2) return launch4<A_MN, B_KC, FA, FB, EPI_INTER16, false, true, kE5M2>(p, s);
        return launch4<A_MN, B_KC, FA, FB, EPI_INTER32, false, true, kF16>(p, s);
      }
    }
  };
};

// MX block scales on 8 waves (A and B both stored k-major, A [K][M] and
// B [K][N]: the 4-wave variant does not fit its registers, which the build
// check would reject), direct cast or fp32 intermediate + cast kernel.
template <bool A_MN, bool B_KC>
struct Mx8Family {
  template <int FA, int FB>
  struct F {
    static hipError_t run(const GemmParams& p, hipStream_t s) {
      if (p.epi == EPI_DIRECT) return launch8<A_MN, B_KC, FA, FB, EPI_DIRECT, false, false, true>(p, s);
      return launch8<A_MN, B_KC, FA, FB, EPI_INTER32, false, false, true>(p, s);
    }
  };
};
constexpr bool mx_on_8_waves(bool a_mn, bool b_kc) { return a_mn && !b_kc; }

}  // namespace scalify
