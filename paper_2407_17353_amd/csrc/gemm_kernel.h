// Scaled FP8 GEMM for gfx950 (MI355X): the FP8 dot_general with fp32
// accumulation of the scaled matmul (Scalify, Section 3.2 / Algorithm 3;
// mixed E4M3/E5M2 inputs and higher-precision accumulation, Appendix A),
// with its epilogue fused: the amax statistic of the dynamic rescale
// (Section 3.3) and either a compact pre-cast intermediate for the cast
// kernel that follows (the dynamic rescale exponent needs the amax of the
// whole output) or, for the delayed rescale, whose output scale is known
// before the GEMM starts, the output codes themselves.
//
// Design (per workgroup: one 256 x 256 output tile, K consumed in 128-byte
// steps, v_mfma_f32_16x16x128_f8f6f4 tiles):
//   * Two wave arrangements (WaveCfg): 4 waves, one per SIMD, each a
//     128 x 128 sub-tile with its 256 accumulators pinned in AGPRs
//     (AccTile), for the plain GEMM whose epilogue stores the pre-cast
//     intermediate; 8 waves, two per SIMD, each a 64 x 128 sub-tile with
//     the accumulators in VGPRs, for the epilogues that convert every value
//     (direct cast, fused add / activation), where the second wave of a
//     SIMD overlaps the first one's arithmetic and stores.
//   * A and B k-slices (32 KiB each per step) stream HBM -> LDS with
//     buffer_load_dwordx4 ... lds (16 B per lane, no VGPR staging) into two
//     64 KiB stages. Buffer loads are range-checked: rows past the matrix,
//     and K past its end, read as zeros without touching memory.
//   * 8 waves: B fragments read from LDS two column groups ahead of their
//     use; one barrier per step, placed before the last quarter of the
//     step's MFMAs: by then every wave holds the B fragments it still
//     needs, so after the barrier the step's stage is free and the loads of
//     step s + 2 are issued into it, two per row block of MFMAs; in the same
//     stretch each wave refills its A fragments with those of step s + 1
//     (landed before the barrier) as soon as their last MFMA has issued.
//   * 4 waves: every B fragment of a step in registers of its own, two
//     barriers per step so that the A and B loads of step s + 2 spread over
//     most of the step (a burst of loads fills the texture address path and
//     stalls the only wave of the SIMD); see the schedule in gemm_kernel.
//   * Operands whose K is contiguous in memory ("KC" tiles, 128 B rows) are
//     read with ds_read_b128; operands whose M or N is contiguous ("MC"
//     tiles, 256 B rows along k) are read with ds_read_b64_tr_b8, which
//     transposes 8x16 byte blocks across 16 lanes, so every storage order
//     feeds the MFMA without a separate transpose pass.
//   * Both tile kinds are XOR-swizzled in 16-byte chunks so that fragment
//     reads hit distinct LDS banks; the swizzle is applied on the global
//     side of the loads because the LDS-direct load writes lane i at
//     M0 + 16 i.
//   * The MFMA is issued with B as its first operand, so each lane ends up
//     holding 4 consecutive output columns: the epilogue stores 8 or 16 byte
//     vectors per lane without an LDS round trip.
//   * Tile order: workgroup ids are remapped so that each XCD (ids are
//     dealt round-robin over the 8 XCDs) walks a contiguous range of tiles,
//     grouped 4 tile-rows high, so the tiles that run together on one XCD
//     share A and B panels in its L2.
#pragma once
#include "codec.h"
#include "kernels.h"

#include <type_traits>

namespace scalify {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int BM = 256, BN = 256, BK = 128;
constexpr int TILE_BYTES = 32768;

// Wave arrangement of a 256 x 256 tile, 2 waves along N:
//   NW = 8: two waves per SIMD, each a 64 x 128 sub-tile (4 x 8 MFMA tiles,
//           accumulators in 128 VGPRs); the two waves of a SIMD cover each
//           other's waits.
//   NW = 4: one wave per SIMD, each a 128 x 128 sub-tile (8 x 8 MFMA tiles,
//           accumulators in 256 AGPRs): a third less LDS traffic per MFMA;
//           every wait of the wave idles its SIMD's matrix core, so its
//           fragments are read a step ahead (A double-buffered).
template <int NW>
struct WaveCfg {
  static constexpr int WAVES = NW, WAVES_N = 2, WAVES_M = NW / 2, NTHR = 64 * NW;
  static constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
  static constexpr int MI = WTM / 16, NI = WTN / 16;
  static constexpr int BPW = 32 / NW;                // 1 KiB load blocks per wave and operand
  static constexpr int LOADS_PER_STEP = 2 * BPW;     // load instructions per wave and step
};

// 16-byte chunk swizzles (see file comment). KC: 16 consecutive rows read
// the same logical chunk from 16 distinct bank groups. MC: the 8 rows a
// 16-lane group reads with one transposing load, and the rows of the
// neighbouring group, fall on distinct chunks.
__device__ __forceinline__ int swz_kc(int r) { return (r & 7) ^ ((r >> 3) & 1); }
__device__ __forceinline__ int swz_mc(int k) { return (k & 7) | (((k >> 5) & 1) << 3); }

// Buffer resource of one operand: base, num_records = bytes of the stored
// matrix, raw (stride 0) gfx9 descriptor word. Loads at offsets >= the
// matrix size return zeros instead of touching memory.
__device__ __forceinline__ v4i make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  v4i r;
  r.x = (int)(uint32_t)a;
  r.y = (int)(uint32_t)(a >> 32);
  r.z = (int)bytes;
  r.w = 0x00020000;
  return r;
}

// One buffer_load_dwordx4 ... lds: lane i's 16 bytes land at M0 + 16 i.
// M0 has no other user in these kernels (no LDS-DMA builtins, no indexed
// register moves), so clobbering it here is safe.
// Issued as inline asm so that the compiler does not order every later LDS
// read behind it; completion is awaited explicitly (wait_vmcnt) before the
// barrier that publishes a k-step.
__device__ __forceinline__ void load_lds16(v4i rsrc, uint32_t voff, uint8_t* lds_base) {
  const uint32_t lds_addr = (uint32_t)(uintptr_t)(LDS_AS void*)lds_base;
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds"
      :
      : "s"(lds_addr), "v"(voff), "s"(rsrc)
      : "memory", "m0");
#pragma clang diagnostic pop
}

// One buffer_load_dword ... lds: lane i's 4 bytes land at M0 + 4 i (the
// MX block-scale staging; same M0 and ordering rules as load_lds16).
__device__ __forceinline__ void load_lds4(v4i rsrc, uint32_t voff, uint8_t* lds_base) {
  const uint32_t lds_addr = (uint32_t)(uintptr_t)(LDS_AS void*)lds_base;
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "buffer_load_dword %1, %2, 0 offen lds"
      :
      : "s"(lds_addr), "v"(voff), "s"(rsrc)
      : "memory", "m0");
#pragma clang diagnostic pop
}

// Wait until at most N of this wave's vector memory loads are outstanding
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most N of this wave's LDS instructions are outstanding
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_lgkmcnt() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}

// Per-thread parts of the chunk offsets of one operand tile. Lane i of a
// wave writes LDS bytes [16 i, 16 i + 16) of its 1 KiB block, so the
// swizzle is applied to the global address; it depends on the lane and on
// the parity of the block, so two lane offsets cover all 8 blocks.
//   KC: tile rows run along M (or N), 128 bytes of K per row; block q of
//       wave w holds rows 8 (8 w + q) .. +7.
//   MC: tile rows run along K, 256 bytes of M (or N) per row; block q of
//       wave w holds k-rows 4 (8 w + q) .. +3.
struct TileLoader {
  uint32_t lane_off[2];  // per parity of the block index
  int kchunk[2];         // KC: k offset (bytes) of the lane's chunk, per parity
};

template <bool KC, int BPW>
__device__ __forceinline__ TileLoader make_loader(uint32_t ld, int wave, int lane) {
  TileLoader L;
  const int hi = ((wave * BPW) >> 3) & 1;  // bit 5 of the k-rows this wave loads (MC)
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    if (KC) {
      const int c = (lane & 7) ^ (lane >> 3) ^ par;
      L.lane_off[par] = (uint32_t)(lane >> 3) * ld + 16u * (uint32_t)c;
      L.kchunk[par] = 16 * c;
    } else {
      const int c = (lane & 15) ^ (par * 4 + (lane >> 4)) ^ (hi << 3);
      L.lane_off[par] = (uint32_t)(lane >> 4) * ld + 16u * (uint32_t)c;
      L.kchunk[par] = 0;
    }
  }
  return L;
}

// Issue chunk load q (0 .. BPW - 1; 1 KiB per wave instruction) of this
// wave's share of one operand tile for the k-step starting at k0.
// Out-of-matrix rows (beyond M or N for KC, beyond K for MC) read zeros
// through the buffer range check; KC chunks that start at or beyond K are
// sent out of range too, and a chunk straddling K is trimmed by
// zero_tail_kc.
// ok = false (no tile left to load: the persistent kernel's last steps)
// sends the whole load out of range.
template <bool KC, int BPW>
__device__ __forceinline__ void issue_block(v4i rsrc, const TileLoader& L, uint32_t ld, int row0,
                                            int k0, int K, uint8_t* lds, int wave, int q,
                                            bool ok = true) {
  const int blk = wave * BPW + q;
  uint32_t off;
  if (KC) {
    off = (uint32_t)(row0 + blk * 8) * ld + (uint32_t)k0 + L.lane_off[q & 1];
    if (k0 + L.kchunk[q & 1] >= K) off = (uint32_t)rsrc.z;
  } else {
    off = (uint32_t)(k0 + blk * 4) * ld + (uint32_t)row0 + L.lane_off[q & 1];
  }
  if (!ok) off = (uint32_t)rsrc.z;
  load_lds16(rsrc, off, lds + blk * 1024);
}

// Origin of output tile t (0 .. tiles_m * tiles_n - 1): ids are dealt
// round-robin over the 8 XCDs, so when the tile count is a multiple of 8,
// id t is remapped so that each XCD walks a contiguous range of tiles; the
// range is walked in groups 4 tile-rows high, so that the tiles that run
// together on one XCD share A and B panels in its L2.
__device__ __forceinline__ void tile_origin(int t, int tiles_m, int tiles_n, int& m0, int& n0) {
  const int T = tiles_m * tiles_n;
  if ((T & 7) == 0) t = (t & 7) * (T >> 3) + (t >> 3);
  constexpr int G = 4;
  const int group = t / (G * tiles_n);
  const int first_m = group * G;
  const int gm = min(tiles_m - first_m, G);
  const int in_group = t - group * G * tiles_n;
  m0 = (first_m + in_group % gm) * BM;
  n0 = (in_group / gm) * BN;
}

// KC tiles when K is not a multiple of 16: zero the bytes k >= krem of the
// chunk that straddles K (chunks wholly beyond K were loaded as zeros).
__device__ __forceinline__ void zero_tail_kc(uint8_t* lds, int krem, int tid) {
  const int r = tid;  // 256 rows, one per thread (threads >= 256 idle)
  if (r >= 256) return;
  const int c = krem >> 4;
  uint8_t* chunk = lds + r * 128 + ((c ^ swz_kc(r)) * 16);
  for (int b = krem & 15; b < 16; ++b) chunk[b] = 0;
}

// 32 k of one row (KC) or one column (MC) of a 16-wide fragment: lane l
// serves row/col (l & 15). The sum over k does not depend on which lane
// holds which k as long as A and B agree, so the plain kernels give lane
// group g = l >> 4 the k = 32 g + 0..31. The MFMA itself orders its 128 k
// as byte j of register half h of lane group g <-> k = 64 h + 16 g + j, and
// its block scale b (from lane group b) covers that order's k 32 b .. + 31;
// block-scaled kernels (HWK) therefore load the fragment in that order.
template <bool KC, bool HWK = false>
__device__ __forceinline__ v8i read_frag(const uint8_t* lds, int base, int lane) {
  v8i f;
  if (KC) {
    const int r = base + (lane & 15);
    const int g = lane >> 4;
    const int s = swz_kc(r);
    const int c0 = HWK ? g : 2 * g, c1 = HWK ? 4 + g : 2 * g + 1;  // 16-byte k chunks
    const v4i lo = *(const v4i*)(lds + r * 128 + ((c0 ^ s) * 16));
    const v4i hi = *(const v4i*)(lds + r * 128 + ((c1 ^ s) * 16));
    f = v8i{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
  } else {
    const int t = lane & 15, g = lane >> 4;
    const int cn = base >> 4;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int k = (HWK ? 64 * (s >> 1) + 16 * g + 8 * (s & 1) : 32 * g + 8 * s) + (t >> 1);
      const int off = k * 256 + ((cn ^ swz_mc(k)) * 16) + (t & 1) * 8;
      const v2i v = __builtin_amdgcn_ds_read_tr8_b64_v2i32((LDS_AS v2i*)(lds + off));
      f[2 * s] = v.x;
      f[2 * s + 1] = v.y;
    }
  }
  return f;
}

template <int FA, int FB>
__device__ __forceinline__ v4f mfma(const v8i& bfrag, const v8i& afrag, const v4f& c) {
  // First operand = B fragment (rows of the MFMA result index N), second =
  // A fragment: result lane l holds C[m = l & 15][n = 4 * (l >> 4) + i].
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(bfrag, afrag, c, FB, FA, 0, 0, 0, 0);
}

// The same MFMA with MX block scales: byte SB of sb and byte SA of sa (E8M0,
// 127 a factor of 1) scale k-block l >> 4 of the step (k 32 (l >> 4) .. + 31
// in the MFMA's k order, which read_frag<..., true> makes the matrix's own)
// of B column / A row (l & 15), for lane l.
template <int FA, int FB, bool MX, int SB = 0, int SA = 0>
__device__ __forceinline__ v4f mfma_s(const v8i& bfrag, const v8i& afrag, const v4f& c, int sb,
                                      int sa) {
  if constexpr (MX)
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(bfrag, afrag, c, FB, FA, SB, sb, SA, sa);
  else
    return mfma<FA, FB>(bfrag, afrag, c);
}

// One LDS read S of a fragment (read_frag split into its instructions, so
// that they can be interleaved one by one with MFMAs): KC parts 0, 1 are
// the two 16-byte halves, MC parts 0 .. 3 the four transposing reads.
template <bool KC, int S, bool HWK = false>
__device__ __forceinline__ void read_frag_part(v8i& f, const uint8_t* lds, int base, int lane) {
  if constexpr (KC) {
    const int r = base + (lane & 15);
    const int g = lane >> 4;
    const int c = HWK ? 4 * S + g : 2 * g + S;  // 16-byte k chunk (read_frag's order)
    const v4i h = *(const v4i*)(lds + r * 128 + ((c ^ swz_kc(r)) * 16));
    f[4 * S + 0] = h.x;
    f[4 * S + 1] = h.y;
    f[4 * S + 2] = h.z;
    f[4 * S + 3] = h.w;
  } else {
    const int t = lane & 15, g = lane >> 4;
    const int k = (HWK ? 64 * (S >> 1) + 16 * g + 8 * (S & 1) : 32 * g + 8 * S) + (t >> 1);
    const int off = k * 256 + (((base >> 4) ^ swz_mc(k)) * 16) + (t & 1) * 8;
    const v2i v = __builtin_amdgcn_ds_read_tr8_b64_v2i32((LDS_AS v2i*)(lds + off));
    f[2 * S] = v.x;
    f[2 * S + 1] = v.y;
  }
}

// Accumulators of the one-wave-per-SIMD GEMM: tile t (t = 8 mi + ni) of a
// wave's 128 x 128 sub-tile lives in AGPRs a[4t .. 4t + 3] for the whole
// main loop, named explicitly in inline asm, so that the compiler, which
// otherwise rotates 256 accumulators through copies and spills, never holds
// or moves them. Every statement declares the AGPRs it writes as clobbered;
// the compiler allocates no AGPR of its own in these kernels (checked on
// the built code object), so nothing else touches them. The compiler does
// not see these MFMAs: their results are read only after mfma_drain().
#define SCALIFY_ACC_TILES(X) \
  X(0, "0:3", "0", "1", "2", "3") \
  X(1, "4:7", "4", "5", "6", "7") \
  X(2, "8:11", "8", "9", "10", "11") \
  X(3, "12:15", "12", "13", "14", "15") \
  X(4, "16:19", "16", "17", "18", "19") \
  X(5, "20:23", "20", "21", "22", "23") \
  X(6, "24:27", "24", "25", "26", "27") \
  X(7, "28:31", "28", "29", "30", "31") \
  X(8, "32:35", "32", "33", "34", "35") \
  X(9, "36:39", "36", "37", "38", "39") \
  X(10, "40:43", "40", "41", "42", "43") \
  X(11, "44:47", "44", "45", "46", "47") \
  X(12, "48:51", "48", "49", "50", "51") \
  X(13, "52:55", "52", "53", "54", "55") \
  X(14, "56:59", "56", "57", "58", "59") \
  X(15, "60:63", "60", "61", "62", "63") \
  X(16, "64:67", "64", "65", "66", "67") \
  X(17, "68:71", "68", "69", "70", "71") \
  X(18, "72:75", "72", "73", "74", "75") \
  X(19, "76:79", "76", "77", "78", "79") \
  X(20, "80:83", "80", "81", "82", "83") \
  X(21, "84:87", "84", "85", "86", "87") \
  X(22, "88:91", "88", "89", "90", "91") \
  X(23, "92:95", "92", "93", "94", "95") \
  X(24, "96:99", "96", "97", "98", "99") \
  X(25, "100:103", "100", "101", "102", "103") \
  X(26, "104:107", "104", "105", "106", "107") \
  X(27, "108:111", "108", "109", "110", "111") \
  X(28, "112:115", "112", "113", "114", "115") \
  X(29, "116:119", "116", "117", "118", "119") \
  X(30, "120:123", "120", "121", "122", "123") \
  X(31, "124:127", "124", "125", "126", "127") \
  X(32, "128:131", "128", "129", "130", "131") \
  X(33, "132:135", "132", "133", "134", "135") \
  X(34, "136:139", "136", "137", "138", "139") \
  X(35, "140:143", "140", "141", "142", "143") \
  X(36, "144:147", "144", "145", "146", "147") \
  X(37, "148:151", "148", "149", "150", "151") \
  X(38, "152:155", "152", "153", "154", "155") \
  X(39, "156:159", "156", "157", "158", "159") \
  X(40, "160:163", "160", "161", "162", "163") \
  X(41, "164:167", "164", "165", "166", "167") \
  X(42, "168:171", "168", "169", "170", "171") \
  X(43, "172:175", "172", "173", "174", "175") \
  X(44, "176:179", "176", "177", "178", "179") \
  X(45, "180:183", "180", "181", "182", "183") \
  X(46, "184:187", "184", "185", "186", "187") \
  X(47, "188:191", "188", "189", "190", "191") \
  X(48, "192:195", "192", "193", "194", "195") \
  X(49, "196:199", "196", "197", "198", "199") \
  X(50, "200:203", "200", "201", "202", "203") \
  X(51, "204:207", "204", "205", "206", "207") \
  X(52, "208:211", "208", "209", "210", "211") \
  X(53, "212:215", "212", "213", "214", "215") \
  X(54, "216:219", "216", "217", "218", "219") \
  X(55, "220:223", "220", "221", "222", "223") \
  X(56, "224:227", "224", "225", "226", "227") \
  X(57, "228:231", "228", "229", "230", "231") \
  X(58, "232:235", "232", "233", "234", "235") \
  X(59, "236:239", "236", "237", "238", "239") \
  X(60, "240:243", "240", "241", "242", "243") \
  X(61, "244:247", "244", "245", "246", "247") \
  X(62, "248:251", "248", "249", "250", "251") \
  X(63, "252:255", "252", "253", "254", "255")

template <int T>
struct AccTile;

// cbsz / blgp select the FP8 formats of the first (B fragment) / second (A
// fragment) operand: 0 E4M3, 1 E5M2.
#define SCALIFY_ACC_TILE(t, r, r0, r1, r2, r3)                                                  \
  template <>                                                                                  \
  struct AccTile<t> {                                                                          \
    /* MX block scales: byte OB of sb (B fragment) and OA of sa (A fragment) */                \
    template <int FA, int FB, int OB, int OA>                                                  \
    static __device__ __forceinline__ void mfma_mx(const v8i& b, const v8i& a, int sb, int sa) { \
      asm volatile("v_mfma_scale_f32_16x16x128_f8f6f4 a[" r "], %0, %1, a[" r "], %2, %3 "     \
                   "op_sel:[%4,%5,0] op_sel_hi:[%6,%7,0] cbsz:%8 blgp:%9"                     \
                   :: "v"(b), "v"(a), "v"(sb), "v"(sa), "n"(OB & 1), "n"(OA & 1), "n"(OB >> 1), \
                      "n"(OA >> 1), "n"(FB), "n"(FA)                                           \
                   : "a" r0, "a" r1, "a" r2, "a" r3);                                          \
    }                                                                                          \
    template <int FA, int FB>                                                                  \
    static __device__ __forceinline__ void mfma(const v8i& b, const v8i& a) {                  \
      if constexpr (FB == 0 && FA == 0)                                                        \
        asm volatile("v_mfma_f32_16x16x128_f8f6f4 a[" r "], %0, %1, a[" r "]"                  \
                     :: "v"(b), "v"(a) : "a" r0, "a" r1, "a" r2, "a" r3);                      \
      else if constexpr (FB == 1 && FA == 0)                                                   \
        asm volatile("v_mfma_f32_16x16x128_f8f6f4 a[" r "], %0, %1, a[" r "] cbsz:1"           \
                     :: "v"(b), "v"(a) : "a" r0, "a" r1, "a" r2, "a" r3);                      \
      else if constexpr (FB == 0 && FA == 1)                                                   \
        asm volatile("v_mfma_f32_16x16x128_f8f6f4 a[" r "], %0, %1, a[" r "] blgp:1"           \
                     :: "v"(b), "v"(a) : "a" r0, "a" r1, "a" r2, "a" r3);                      \
      else                                                                                     \
        asm volatile("v_mfma_f32_16x16x128_f8f6f4 a[" r "], %0, %1, a[" r "] cbsz:1 blgp:1"    \
                     :: "v"(b), "v"(a) : "a" r0, "a" r1, "a" r2, "a" r3);                      \
    }                                                                                          \
    static __device__ __forceinline__ void zero() {                                            \
      asm volatile("v_accvgpr_write_b32 a" r0 ", 0\n\tv_accvgpr_write_b32 a" r1 ", 0\n\t"       \
                   "v_accvgpr_write_b32 a" r2 ", 0\n\tv_accvgpr_write_b32 a" r3 ", 0"          \
                   ::: "a" r0, "a" r1, "a" r2, "a" r3);                                        \
    }                                                                                          \
    static __device__ __forceinline__ v4f read() {                                             \
      float x0, x1, x2, x3;                                                                    \
      asm volatile("v_accvgpr_read_b32 %0, a" r0 "\n\tv_accvgpr_read_b32 %1, a" r1 "\n\t"      \
                   "v_accvgpr_read_b32 %2, a" r2 "\n\tv_accvgpr_read_b32 %3, a" r3               \
                   : "=v"(x0), "=v"(x1), "=v"(x2), "=v"(x3));                                  \
      return v4f{x0, x1, x2, x3};                                                              \
    }                                                                                          \
  };
SCALIFY_ACC_TILES(SCALIFY_ACC_TILE)
#undef SCALIFY_ACC_TILE

// Wait states after the last AccTile write before its registers are read by
// other instructions (more than the 8-pass MFMA's result latency).
__device__ __forceinline__ void mfma_drain() {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Direct cast of 4 pre-cast values (fp32 bits) times 2^-shift, for the
// delayed rescale. Fast paths use the hardware conversions (callers check
// that the shift is in their exact window and that no value is NaN); the
// exact integer casts are kept out of line.
__device__ __forceinline__ v2i cast4_f16_hw(uint32_t u0, uint32_t u1, uint32_t u2, uint32_t u3,
                                           float inv, bool sat) {
  // x * 2^-shift (inv = 2^-shift) is exact in fp32 unless it leaves the
  // fp32 normal range: above it the conversion overflows as the exact value
  // would, below it the value rounds to zero in FP16 either way.
  // v_cvt_f16_f32 then rounds to nearest even, keeping FP16 subnormals;
  // overflow gives Inf, which saturation turns into max. The magnitude is
  // converted and the sign put back: the compiler fuses the multiply and
  // the conversion into an fma whose +0 addend would turn -0 into +0.
  uint32_t h[4];
  const uint32_t u[4] = {u0, u1, u2, u3};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const _Float16 f = (_Float16)(__uint_as_float(u[i] & 0x7FFFFFFFu) * inv);
    uint32_t b = (uint32_t)__builtin_bit_cast(uint16_t, f);
    if (sat && b == 0x7C00u) b = 0x7BFFu;  // Inf -> 65504
    h[i] = b | ((u[i] >> 16) & 0x8000u);
  }
  return v2i{(int)(h[0] | (h[1] << 16)), (int)(h[2] | (h[3] << 16))};
}

__device__ __attribute__((noinline)) v2i cast4_slow_f16(uint32_t u0, uint32_t u1, uint32_t u2,
                                                         uint32_t u3, int shift, bool sat) {
  return v2i{(int)(cast_bits<kF16>(u0, shift, sat) | (cast_bits<kF16>(u1, shift, sat) << 16)),
             (int)(cast_bits<kF16>(u2, shift, sat) | (cast_bits<kF16>(u3, shift, sat) << 16))};
}

__device__ __attribute__((noinline)) uint32_t cast4_slow_fp8(int fmt, uint32_t u0, uint32_t u1,
                                                              uint32_t u2, uint32_t u3, int shift,
                                                              bool sat) {
  if (fmt == kE4M3)
    return cast_bits<kE4M3>(u0, shift, sat) | (cast_bits<kE4M3>(u1, shift, sat) << 8) |
           (cast_bits<kE4M3>(u2, shift, sat) << 16) | (cast_bits<kE4M3>(u3, shift, sat) << 24);
  return cast_bits<kE5M2>(u0, shift, sat) | (cast_bits<kE5M2>(u1, shift, sat) << 8) |
         (cast_bits<kE5M2>(u2, shift, sat) << 16) | (cast_bits<kE5M2>(u3, shift, sat) << 24);
}

// ---- fused epilogue: scaled add of a residual (Algorithm 3 rule) and an
// activation f(x) = x * g(x) with the scale kept (Appendix C.1).

// Raw residual codes at row m, columns n..n+3 (columns >= N are not read
// and come back as 0): FP8 packs the 4 codes in c[0], FP16 two per word.
__device__ __forceinline__ void load_residual_codes(const GemmParams& p, int m, int n,
                                                    uint32_t (&c)[2]) {
  const int64_t e = (int64_t)m * p.ldr + n;
  c[0] = c[1] = 0u;
  if (p.res_fmt == kF16) {
    const uint16_t* q = (const uint16_t*)p.res + e;
    if (n + 3 < p.N) {
      const v2i w = *(const v2i*)q;
      c[0] = (uint32_t)w.x;
      c[1] = (uint32_t)w.y;
    } else {
      c[0] = q[0];
      if (n + 1 < p.N) c[0] |= (uint32_t)q[1] << 16;
      if (n + 2 < p.N) c[1] = q[2];
    }
  } else {
    const uint8_t* q = (const uint8_t*)p.res + e;
    if (n + 3 < p.N) {
      c[0] = *(const uint32_t*)q;
    } else {
      c[0] = q[0];
      if (n + 1 < p.N) c[0] |= (uint32_t)q[1] << 8;
      if (n + 2 < p.N) c[0] |= (uint32_t)q[2] << 16;
    }
  }
}

// Residual codes decoded to fp32 (exact: every FP8 and FP16 value is an
// fp32) by the hardware conversions, OCP FP8 with a unit scale.
__device__ __forceinline__ v4f decode_residual4(int fmt, uint32_t c0, uint32_t c1) {
  v4f r;
  if (fmt == kF16) {
    r[0] = (float)__builtin_bit_cast(_Float16, (uint16_t)(c0 & 0xFFFFu));
    r[1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(c0 >> 16));
    r[2] = (float)__builtin_bit_cast(_Float16, (uint16_t)(c1 & 0xFFFFu));
    r[3] = (float)__builtin_bit_cast(_Float16, (uint16_t)(c1 >> 16));
  } else if (fmt == kE4M3) {
    r[0] = __builtin_amdgcn_cvt_scalef32_f32_fp8(c0, 1.0f, 0);
    r[1] = __builtin_amdgcn_cvt_scalef32_f32_fp8(c0, 1.0f, 1);
    r[2] = __builtin_amdgcn_cvt_scalef32_f32_fp8(c0, 1.0f, 2);
    r[3] = __builtin_amdgcn_cvt_scalef32_f32_fp8(c0, 1.0f, 3);
  } else {
    r[0] = __builtin_amdgcn_cvt_scalef32_f32_bf8(c0, 1.0f, 0);
    r[1] = __builtin_amdgcn_cvt_scalef32_f32_bf8(c0, 1.0f, 1);
    r[2] = __builtin_amdgcn_cvt_scalef32_f32_bf8(c0, 1.0f, 2);
    r[3] = __builtin_amdgcn_cvt_scalef32_f32_bf8(c0, 1.0f, 3);
  }
  return r;
}

// Smooth gates in fp32: silu g(x) = 1 / (1 + e^-x); the tanh form of gelu
// (1 + tanh(u)) / 2 with u = sqrt(2/pi) (x + 0.044715 x^3) is the same
// sigmoid at 2u. Both are 1 and 0 at +-Inf and NaN for NaN, within a few
// ulp of the exact gate where it is a normal fp32 (below 2^-126 it may
// flush to 0).
template <bool GELU>
__device__ __forceinline__ float smooth_gate(float x) {
  const float k0 = 1.5957691216057308f;   // 2 sqrt(2/pi)
  const float k1 = 0.07135481627260025f;  // 2 sqrt(2/pi) * 0.044715
  const float t = GELU ? x * (k0 + k1 * (x * x)) : x;
  return __builtin_amdgcn_rcpf(1.0f + expf(-t));
}

// The fused pre-cast values of a wave's accumulators, in place: the scaled
// add of the residual (format RF; power-of-two shifts sh_acc and sh_res into
// w's scale 2^e_w), then the activation ACT, whose gate sees the true value
// w * 2^e_w. One straight pass per transformation. The residual codes of all
// the wave's outputs are loaded first, so that their latencies overlap; a
// wave tile inside the matrix loads them without per-output checks.
// Exponent of a power of two held in fp32 (normal or subnormal encoding).
__device__ __forceinline__ int pow2_exponent_of(float x) {
  const uint32_t u = __float_as_uint(x);
  const int e = (int)((u >> 23) & 0xFFu);
  if (e != 0) return e - 127;
  const uint32_t m = u & 0x7FFFFFu;
  return m ? (31 - __clz((int)m)) - 149 : -127;
}

// Channel exponents of a wave's outputs, packed 4 to a register as e + 128
// (channel scales lie in the E8M0 range [2^-127, 2^127]): cha[mi] for the
// row block (rows mb + 16 mi), chb[ni] byte i for column nb + 16 ni + i; 0
// where there is no channel scale or the output lies outside the matrix.
// All loads are issued before the first use; the packed form keeps the
// registers free for the residual codes loaded next.
template <int MI_, int NI_>
__device__ __forceinline__ void load_channel_exponents(const GemmParams& p, int mb, int nb,
                                                       int (&cha)[MI_], uint32_t (&chb)[NI_]) {
  float va[MI_];
  v4f vb[NI_];
#pragma unroll
  for (int mi = 0; mi < MI_; ++mi) {
    const int m = mb + 16 * mi;
    va[mi] = (p.ch_a && m < p.M) ? p.ch_a[m] : 1.0f;
  }
#pragma unroll
  for (int ni = 0; ni < NI_; ++ni) {
    const int n = nb + 16 * ni;
    if (p.ch_b && n + 3 < p.N) {
      vb[ni] = *(const v4f*)(p.ch_b + n);
    } else {
      vb[ni] = v4f{1.f, 1.f, 1.f, 1.f};
      if (p.ch_b) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (n + i < p.N) vb[ni][i] = p.ch_b[n + i];
      }
    }
  }
#pragma unroll
  for (int mi = 0; mi < MI_; ++mi) cha[mi] = pow2_exponent_of(va[mi]);
#pragma unroll
  for (int ni = 0; ni < NI_; ++ni) {
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) w |= (uint32_t)(pow2_exponent_of(vb[ni][i]) + 128) << (8 * i);
    chb[ni] = w;
  }
}

__device__ __forceinline__ int chb_exp(uint32_t packed, int i) {
  return (int)((packed >> (8 * i)) & 0xFFu) - 128;
}

template <int RF, bool CH, int MI_, int NI_>
__device__ __forceinline__ void add_residual(const GemmParams& p, v4f (&acc)[MI_][NI_], int mb,
                                             int nb, bool interior, int sh_acc, int sh_res,
                                             const int (&cha)[MI_], const uint32_t (&chb)[NI_]) {
  constexpr int W = RF == kF16 ? 2 : 1;  // code words per 4 outputs
  uint32_t rc[MI_][NI_][W];
  if (interior) {
    static_for<0, MI_ * NI_>([&](auto I) {
      constexpr int mi = decltype(I)::value / NI_, ni = decltype(I)::value % NI_;
      const int64_t e = (int64_t)(mb + 16 * mi) * p.ldr + nb + 16 * ni;
      if constexpr (RF == kF16) {
        const v2i w = *(const v2i*)((const uint16_t*)p.res + e);
        rc[mi][ni][0] = (uint32_t)w.x;
        rc[mi][ni][W - 1] = (uint32_t)w.y;
      } else {
        rc[mi][ni][0] = *(const uint32_t*)((const uint8_t*)p.res + e);
      }
    });
  } else {
    static_for<0, MI_ * NI_>([&](auto I) {
      constexpr int mi = decltype(I)::value / NI_, ni = decltype(I)::value % NI_;
      const int m = mb + 16 * mi;
      const int n = nb + 16 * ni;
      uint32_t c[2] = {0u, 0u};
      if (m < p.M && n < p.N) load_residual_codes(p, m, n, c);
      rc[mi][ni][0] = c[0];
      rc[mi][ni][W - 1] = RF == kF16 ? c[1] : c[0];
    });
  }
  static_for<0, MI_ * NI_>([&](auto I) {
    constexpr int mi = decltype(I)::value / NI_, ni = decltype(I)::value % NI_;
    const v4f r = decode_residual4(RF, rc[mi][ni][0], rc[mi][ni][W - 1]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      acc[mi][ni][i] = ldexpf(acc[mi][ni][i], CH ? sh_acc + cha[mi] + chb_exp(chb[ni], i) : sh_acc) +
                       ldexpf(r[i], sh_res);
    __builtin_amdgcn_sched_barrier(0);  // one group at a time: bounded register use
  });
}

template <int ACT, int MI_, int NI_>
__device__ __forceinline__ void activate(v4f (&acc)[MI_][NI_], int e_w) {
  static_for<0, MI_ * NI_>([&](auto I) {
    constexpr int mi = decltype(I)::value / NI_, ni = decltype(I)::value % NI_;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float v = acc[mi][ni][i];
      if constexpr (ACT == ACT_RELU) {
        acc[mi][ni][i] = v * (v > 0.0f ? 1.0f : 0.0f);
      } else {
        acc[mi][ni][i] = v * smooth_gate<ACT == ACT_GELU_TANH>(ldexpf(v, e_w));
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // one group at a time: bounded register use
  });
}

// CH: the fused epilogue also applies channel scales (instantiated apart, so
// that the other fused kernels keep their register allocation).
template <bool A_MN, bool B_KC, int FA, int FB, int EPI, bool FUSE, int NW, bool CH = false,
          bool MX = false>
__global__ __launch_bounds__(64 * NW, 1) void gemm_kernel(GemmParams p) {
  static_assert(NW == 8, "two waves per SIMD (the 4-wave arrangement is gemm4_kernel)");
  static_assert(FUSE || !CH, "channel scales are part of the fused epilogue");
  static_assert(!MX || (!FUSE && (EPI == EPI_INTER32 || EPI == EPI_DIRECT)),
                "block scales: plain epilogue, fp32 intermediate or direct cast");
  using C = WaveCfg<NW>;
  constexpr int WAVES = C::WAVES, WAVES_N = C::WAVES_N, WTM = C::WTM, WTN = C::WTN;
  constexpr int MI = C::MI, NI = C::NI, BPW = C::BPW, LOADS_PER_STEP = C::LOADS_PER_STEP;
  __shared__ __attribute__((aligned(1024))) uint8_t sA0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sB0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sB1[TILE_BYTES];
  __shared__ float red[WAVES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  int m0, n0;
  tile_origin(blockIdx.x, p.tiles_m, p.tiles_n, m0, n0);

  const int M = p.M, N = p.N, K = p.K;
  const int KT = (K + BK - 1) / BK;
  const int KT_full = K / BK;         // k-steps entirely inside K
  const int krem = K - KT_full * BK;  // bytes of the partial last step (0 if none)
  const uint32_t lda = (uint32_t)p.lda, ldb = (uint32_t)p.ldb;

  // A: KC when stored [M][K], MC when stored [K][M] (row0 = m0 either way).
  // B: KC when stored [N][K], MC when stored [K][N].
  const v4i ra = make_rsrc(p.a, p.a_bytes);
  const v4i rb = make_rsrc(p.b, p.b_bytes);
  const TileLoader la = make_loader<!A_MN, BPW>(lda, wave, lane);
  const TileLoader lb = make_loader<B_KC, BPW>(ldb, wave, lane);

  // Load j of a step: j < BPW are A blocks, the rest B blocks.
  auto issue_one = [&](int j, int kt, uint8_t* dA, uint8_t* dB) {
    if (j < BPW)
      issue_block<!A_MN, BPW>(ra, la, lda, m0, kt * BK, K, dA, wave, j);
    else
      issue_block<B_KC, BPW>(rb, lb, ldb, n0, kt * BK, K, dB, wave, j - BPW);
  };
  auto issue_all = [&](int kt, uint8_t* dA, uint8_t* dB) {
#pragma unroll
    for (int j = 0; j < LOADS_PER_STEP; ++j) issue_one(j, kt, dA, dB);
  };
  // The partial last step's stage, once landed: clear the KC bytes >= K.
  auto zero_tail = [&](uint8_t* dA, uint8_t* dB) {
    if (!A_MN) zero_tail_kc(dA, krem, tid);
    if (B_KC) zero_tail_kc(dB, krem, tid);
    __syncthreads();
  };

  // MX block scales, packed (see GemmParams): a k-step's 256 bytes of one
  // 64-row group are contiguous, so wave w < 4 stages A's group m0 / 64 + w
  // and wave w >= 4 B's group n0 / 64 + w - 4 with one 256-byte load beside
  // the step's tiles (groups past the array read zeros: rows past M or N,
  // whose data are zero). Stage layout: [2 k-step stages][A 1 KiB | B 1 KiB],
  // tile group j at 256 j. Lane l's word of a group holds the bytes of its
  // 4 row blocks (rows l & 15, + 16, + 32, + 48) at k-block l >> 4.
  uint8_t* sS = nullptr;
  if constexpr (MX) {
    __shared__ __attribute__((aligned(1024))) uint8_t s_mx[4096];
    sS = s_mx;
  }
  // 4 waves: wave w stages group w of A (half 0) and of B (half 1), one call each.
  auto issue_scale_half = [&](int kt, int stage, bool is_b) {
    if constexpr (MX) {
      const int groups = is_b ? p.mx_groups_b : p.mx_groups_a;
      const int grp = (is_b ? n0 : m0) / 64 + wave;
      const v4i r = is_b ? make_rsrc(p.mx_b, p.mx_b_bytes) : make_rsrc(p.mx_a, p.mx_a_bytes);
      const uint32_t off =
          grp < groups ? ((uint32_t)(kt * groups + grp) * 64u + (uint32_t)lane) * 4u : (uint32_t)r.z;
      load_lds4(r, off, sS + stage * 2048 + (is_b ? 1024 : 0) + 256 * wave);
    }
  };
  auto issue_scales = [&](int kt, int stage) {
    if constexpr (MX) {
      const bool is_b = wave >= 4;
      const int groups = is_b ? p.mx_groups_b : p.mx_groups_a;
      const int grp = (is_b ? n0 : m0) / 64 + (wave & 3);
      const v4i r = is_b ? make_rsrc(p.mx_b, p.mx_b_bytes) : make_rsrc(p.mx_a, p.mx_a_bytes);
      const uint32_t off =
          grp < groups ? ((uint32_t)(kt * groups + grp) * 64u + (uint32_t)lane) * 4u : (uint32_t)r.z;
      load_lds4(r, off, sS + stage * 2048 + (is_b ? 1024 : 0) + 256 * (wave & 3));
    }
  };
  // This lane's word of tile group j (0..3) of operand half (0 A, 1 B).
  auto scale_word = [&](int stage, int half, int j) -> int {
    return *(const int*)(sS + stage * 2048 + half * 1024 + 256 * j + 4 * lane);
  };

  v4f acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  const int wm = (wave / WAVES_N) * WTM;  // wave sub-tile
  const int wn = (wave % WAVES_N) * WTN;
  constexpr int DSA = A_MN ? 4 : 2;  // LDS reads per A fragment
  constexpr int DSB = B_KC ? 2 : 4;  // LDS reads per B fragment
  static_assert(LOADS_PER_STEP == 2 * MI, "two loads per row block");
  using T_ = std::true_type;
  using F_ = std::false_type;

  {
    v8i a[MI];   // A fragments of the step
    v8i bq[3];   // B fragments: in use and up to two groups ahead
    // MX: this lane's block-scale words of the step: A's for the wave's 64
    // rows (byte mi), B's for its column groups 0 .. 3 and 4 .. 7 (byte ni & 3)
    int sa = 0, sb[2] = {0, 0};
    static_assert(!MX || (MI == 4 && NI == 8 && WTM == 64 && WTN == 128), "MX word layout");

    // One k-step. LOADS: issue the loads of step kt + 2 into this step's
    // stage after the barrier. NEXT: step kt + 1 exists (barrier, then its A
    // fragments and first B fragment are read into a[] and b).
    auto step = [&](auto loads_tag, auto next_tag, int kt) {
      constexpr bool LOADS = decltype(loads_tag)::value;
      constexpr bool NEXT = decltype(next_tag)::value;
      const bool odd = kt & 1;
      uint8_t* cA = odd ? sA1 : sA0;  // this step's stage
      uint8_t* cB = odd ? sB1 : sB0;
      uint8_t* nA = odd ? sA0 : sA1;  // the next step's stage
      uint8_t* nB = odd ? sB0 : sB1;
      // B column groups 0 .. NI - 3, fragments read two groups ahead
      static_for<0, NI - 2>([&](auto I) {
        constexpr int ni = decltype(I)::value;
        bq[(ni + 2) % 3] = read_frag<B_KC, MX>(cB, wn + 16 * (ni + 2), lane);
        static_for<0, MI>([&](auto J) {
          constexpr int mi = decltype(J)::value;
          acc[mi][ni] =
              mfma_s<FA, FB, MX, ni & 3, mi>(bq[ni % 3], a[mi], acc[mi][ni], sb[ni >> 2], sa);
        });
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          if (mi < DSB) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      });
      if (NEXT) {
        // Every wave holds all B fragments of this step once its LDS reads
        // have returned (the barrier waits for them), so this stage is free
        // after the barrier; step kt + 1 has landed once every wave's loads
        // have completed.
        wait_vmcnt<0>();
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
        if (!LOADS && kt + 1 == KT_full && (krem & 15)) zero_tail(nA, nB);
        // MX: B column groups 0 .. 3 are done with their word
        if constexpr (MX) sb[0] = scale_word(!odd, 1, wn / 64);
      }
      // B column groups NI - 2 and NI - 1, taken row block by row block: once
      // both MFMAs of a[mi] have issued, a[mi] is refilled with the fragment
      // of step kt + 1; the loads of step kt + 2 go out two per row block.
      static_for<0, MI>([&](auto J) {
        constexpr int mi = decltype(J)::value;
        acc[mi][NI - 2] = mfma_s<FA, FB, MX, (NI - 2) & 3, mi>(bq[(NI - 2) % 3], a[mi],
                                                                acc[mi][NI - 2], sb[1], sa);
        acc[mi][NI - 1] = mfma_s<FA, FB, MX, (NI - 1) & 3, mi>(bq[(NI - 1) % 3], a[mi],
                                                                acc[mi][NI - 1], sb[1], sa);
        if (LOADS) {
          issue_one(2 * mi, kt + 2, cA, cB);
          issue_one(2 * mi + 1, kt + 2, cA, cB);
          if (mi == MI - 1) issue_scales(kt + 2, odd);
        }
        if (NEXT) a[mi] = read_frag<!A_MN, MX>(nA, wm + 16 * mi, lane);
      });
      if (NEXT) {
        bq[0] = read_frag<B_KC, MX>(nB, wn, lane);
        bq[1] = read_frag<B_KC, MX>(nB, wn + 16, lane);
        if constexpr (MX) {  // every MFMA of this step has issued
          sb[1] = scale_word(!odd, 1, wn / 64 + 1);
          sa = scale_word(!odd, 0, wm / 64);
        }
      }
      static_for<0, MI>([&](auto I) {
        constexpr int i = decltype(I)::value;
        // MX: one B word after the barrier, a B and the A word at the end
        constexpr int XS = MX ? (i == 0 ? 1 : 0) + (i + 1 == MI ? 2 : 0) : 0;
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        if (NEXT)
          __builtin_amdgcn_sched_group_barrier(0x100, (i + 1 < MI ? DSA : DSA + 2 * DSB) + XS, 0);
      });
    };

    if (KT > 0) {
      issue_all(0, sA0, sB0);
      issue_scales(0, 0);
      if (KT > 1) {
        issue_all(1, sA1, sB1);
        issue_scales(1, 1);
        wait_vmcnt<LOADS_PER_STEP + (MX ? 1 : 0)>();  // step 1's loads may be in flight
      } else {
        wait_vmcnt<0>();
      }
      __syncthreads();
      if (KT_full == 0 && (krem & 15)) zero_tail(sA0, sB0);
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) a[mi] = read_frag<!A_MN, MX>(sA0, wm + 16 * mi, lane);
      bq[0] = read_frag<B_KC, MX>(sB0, wn, lane);
      bq[1] = read_frag<B_KC, MX>(sB0, wn + 16, lane);
      if constexpr (MX) {
        sa = scale_word(0, 0, wm / 64);
        sb[0] = scale_word(0, 1, wn / 64);
        sb[1] = scale_word(0, 1, wn / 64 + 1);
      }
    }
    int kt = 0;
    for (; kt + 2 < KT; ++kt) step(T_{}, T_{}, kt);
    if (kt + 1 < KT) step(F_{}, T_{}, kt++);
    if (kt < KT) step(F_{}, F_{}, kt);
  }

  // ---- epilogue: lane holds C[m][n..n+3] for each (mi, ni)
  float lmax = 0.f;
  const int mb = m0 + wm + (lane & 15);
  const int nb = n0 + wn + 4 * (lane >> 4);
  // EPI_DIRECT: data' = acc * 2^-shift, shift from the prologue
  const int shift = EPI == EPI_DIRECT ? (int)__builtin_amdgcn_readfirstlane(p.hdr[2]) : 0;
  // Fused values and block-scaled accumulators may be fp32 subnormals (the
  // plain accumulators never are).
  const bool fast =
      shift >= ((FUSE || MX) ? kFastShiftMinSub : -kFastShiftMax) && shift <= kFastShiftMax;
  const float hw_scale = fast ? pow2_float(shift) : 1.0f;
  const float hw_inv = fast ? pow2_float(-shift) : 1.0f;
  const bool sat = p.sat != 0;
  // FUSE: a first pass turns every accumulator into its pre-cast value w
  // (scaled add, activation) before any store is issued, so that the only
  // memory waits are those of the residual codes, all loaded up front; the
  // pass below then writes w as the plain epilogue writes acc.
  if constexpr (FUSE) {
    const int e_w = (int)__builtin_amdgcn_readfirstlane(p.hdr[1]);
    if (p.acc_out) {
      static_for<0, MI * NI>([&](auto I) {
        constexpr int mi = decltype(I)::value / NI, ni = decltype(I)::value % NI;
        const int m = mb + 16 * mi;
        const int n = nb + 16 * ni;
        if (m < M && n < N) {
          const v4f a = acc[mi][ni];
          float* q = p.acc_out + (int64_t)m * N + n;
          q[0] = a[0];
          if (n + 1 < N) q[1] = a[1];
          if (n + 2 < N) q[2] = a[2];
          if (n + 3 < N) q[3] = a[3];
        }
      });
    }
    // Channel scales (CH): one power-of-two product of the accumulator,
    // folded into the scaled add's shift when there is a residual.
    int cha[MI] = {};
    uint32_t chb[NI] = {};
    if constexpr (CH) {
      load_channel_exponents(p, mb, nb, cha, chb);
      __builtin_amdgcn_sched_barrier(0);
    } else {
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) chb[ni] = 0x80808080u;  // exponent 0
    }
    if (p.res) {
      const bool interior = m0 + wm + 16 * MI <= M && n0 + wn + 16 * NI <= N;
      const int sh_acc = (int)__builtin_amdgcn_readfirstlane(p.hdr[3]);
      const int sh_res = (int)__builtin_amdgcn_readfirstlane(p.hdr[4]);
      if (p.res_fmt == kE4M3) add_residual<kE4M3, CH>(p, acc, mb, nb, interior, sh_acc, sh_res, cha, chb);
      else if (p.res_fmt == kE5M2) add_residual<kE5M2, CH>(p, acc, mb, nb, interior, sh_acc, sh_res, cha, chb);
      else add_residual<kF16, CH>(p, acc, mb, nb, interior, sh_acc, sh_res, cha, chb);
    } else if constexpr (CH) {
      static_for<0, MI * NI>([&](auto I) {
        constexpr int mi = decltype(I)::value / NI, ni = decltype(I)::value % NI;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[mi][ni][i] = ldexpf(acc[mi][ni][i], cha[mi] + chb_exp(chb[ni], i));
      });
    }
    if (p.act == ACT_RELU) activate<ACT_RELU>(acc, e_w);
    else if (p.act == ACT_GELU_TANH) activate<ACT_GELU_TANH>(acc, e_w);
    else if (p.act == ACT_SILU) activate<ACT_SILU>(acc, e_w);
  }
  static_for<0, MI * NI>([&](auto I) {
    constexpr int mi = decltype(I)::value / NI, ni = decltype(I)::value % NI;
    const int m = mb + 16 * mi;
    const int n = nb + 16 * ni;
    if (m < M && n < N) {
      const v4f v = acc[mi][ni];  // FUSE: w
      lmax = fmaxf(lmax, fabsf(v[0]));
      if (n + 1 < N) lmax = fmaxf(lmax, fabsf(v[1]));
      if (n + 2 < N) lmax = fmaxf(lmax, fabsf(v[2]));
      if (n + 3 < N) lmax = fmaxf(lmax, fabsf(v[3]));
      if (EPI == EPI_INTER16) {
        const uint32_t h0 = sticky16(__float_as_uint(v[0])), h1 = sticky16(__float_as_uint(v[1]));
        const uint32_t h2 = sticky16(__float_as_uint(v[2])), h3 = sticky16(__float_as_uint(v[3]));
        uint16_t* q = (uint16_t*)p.inter + (int64_t)m * p.ldw + n;
        *(v2i*)q = v2i{(int)(h0 | (h1 << 16)), (int)(h2 | (h3 << 16))};
      } else if (EPI == EPI_INTER32) {
        float* q = (float*)p.inter + (int64_t)m * p.ldw + n;
        *(v4f*)q = v;
      } else {
        const uint32_t u0 = __float_as_uint(v[0]), u1 = __float_as_uint(v[1]);
        const uint32_t u2 = __float_as_uint(v[2]), u3 = __float_as_uint(v[3]);
        // Hardware conversions unless a lane of the wave holds a NaN or the
        // shift is out of their range (then the exact integer cast, out of
        // line: it is rare and large).
        const bool nan = is_nan_bits(u0) || is_nan_bits(u1) || is_nan_bits(u2) || is_nan_bits(u3);
        const bool hw = fast && !__any(nan);
        if (p.out_fmt == kF16) {
          v2i w;
          if (hw) {
            w = cast4_f16_hw(u0, u1, u2, u3, hw_inv, sat);
          } else {
            w = cast4_slow_f16(u0, u1, u2, u3, shift, sat);
          }
          uint16_t* q = (uint16_t*)p.out + (int64_t)m * p.ldc + n;
          if (n + 3 < N) {
            *(v2i*)q = w;
          } else {
            q[0] = (uint16_t)w.x;
            if (n + 1 < N) q[1] = (uint16_t)((uint32_t)w.x >> 16);
            if (n + 2 < N) q[2] = (uint16_t)w.y;
          }
        } else {
          uint32_t w;
          if (hw) {
            w = p.out_fmt == kE4M3 ? cast4_fp8_hw<kE4M3>(u0, u1, u2, u3, hw_scale, sat)
                                   : cast4_fp8_hw<kE5M2>(u0, u1, u2, u3, hw_scale, sat);
          } else {
            w = cast4_slow_fp8(p.out_fmt, u0, u1, u2, u3, shift, sat);
          }
          uint8_t* q = (uint8_t*)p.out + (int64_t)m * p.ldc + n;
          if (n + 3 < N) {
            *(uint32_t*)q = w;
          } else {
            q[0] = (uint8_t)w;
            if (n + 1 < N) q[1] = (uint8_t)(w >> 8);
            if (n + 2 < N) q[2] = (uint8_t)(w >> 16);
          }
        }
      }
      if (!FUSE && p.acc_out) {
        const v4f a = v;
        float* q = p.acc_out + (int64_t)m * N + n;
        q[0] = a[0];
        if (n + 1 < N) q[1] = a[1];
        if (n + 2 < N) q[2] = a[2];
        if (n + 3 < N) q[3] = a[3];
      }
      if constexpr (FUSE) {
        if (p.pre_out) {
          float* q = p.pre_out + (int64_t)m * N + n;
          q[0] = v[0];
          if (n + 1 < N) q[1] = v[1];
          if (n + 2 < N) q[2] = v[2];
          if (n + 3 < N) q[3] = v[3];
        }
      }
    }
  });
  // amax of |acc| over the valid elements (fmaxf ignores NaN): wave
  // butterfly, then across the waves, then one atomic max per workgroup
  // on the fp32 bits (non-negative floats order like their bits).
  for (int off = 32; off > 0; off >>= 1) lmax = fmaxf(lmax, __shfl_xor(lmax, off, 64));
  if (lane == 0) red[wave] = lmax;
  __syncthreads();
  if (tid == 0) {
    float wmax = red[0];
    for (int w = 1; w < WAVES; ++w) wmax = fmaxf(wmax, red[w]);
    atomicMax(p.hdr, __float_as_uint(wmax));
  }
}

}  // namespace scalify
