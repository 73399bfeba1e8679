// Causal sliding-window attention (MegaScale Section 3.1, "Sliding window
// attention"), evaluated flash-style as Section 3.3 adopts FlashAttention-2:
// scores never reach HBM, softmax is computed online, and key tiles that lie
// wholly outside a query block's window are never visited, so the work is
// O(seq * window).  Query i sees key j iff 0 <= i - j < window.
//
// bf16 kernels (gfx950 MFMA 32x32x16).  Everything is computed transposed:
// the MFMA's "A" operand is the key (or d) side, so the 32 output columns a
// lane owns are 32 queries (forward, dQ) or 32 keys (dK/dV).  Each lane then
// holds all scores of ONE query; the softmax rescale is a per-lane scalar,
// the row maximum needs a single cross-half exchange, and the probabilities
// feed the next MFMA straight from the accumulator registers (the k-index
// order of that MFMA is permuted to match, and the LDS copy of the other
// operand is written in the same permuted order).
//   forward : S^T = K Q^T, O^T += V^T P^T         (LDS: K, V^T)
//   dK, dV  : S = Q K^T, dP = dO V^T,
//             dV^T += dO^T P, dK^T += Q^T dS       (LDS: Q, Q^T, dO, dO^T)
//   dQ      : S^T = K Q^T, dP^T = V dO^T,
//             dQ^T += K^T dS^T                     (LDS: K, K^T, V)
// The backward pass is split in two kernels so that no gradient needs atomic
// accumulation: results are deterministic.
//
// fp32 kernels: one thread per query (or key), plain loops; parity path.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace pb {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();

// Waves per workgroup and tile length (tokens per LDS tile):
//   forward and dQ: 32 kWavesQ queries per workgroup, key tiles of kTL
//   dK/dV         : kBlockK keys per workgroup (kWavesK waves), query tiles of kTLdkv
// Four forward / dQ waves share each K/V tile, which with two workgroups per
// CU (64 KB of LDS each) keeps two waves on every SIMD, so one wave's
// softmax arithmetic overlaps another's matrix instructions.
constexpr int kWavesQ = 4;
constexpr int kWavesK = 4;  // two key groups of 32, each with a P wave and a dS wave
constexpr int kTL = 64;      // forward and dQ key tiles
constexpr int kTLdkv = 32;   // dK/dV query tiles (keeps its registers and LDS in budget)
constexpr int kStagesDkdv = 4;  // dK/dV LDS stages: tile loads run three tiles ahead
constexpr int kBlockQ = 32 * kWavesQ;  // queries per forward / dQ workgroup
constexpr int kBlockK = 64;            // keys per dK/dV workgroup
constexpr int kUnsplit = 1 << 30;

// Key tiles (of kTL) that the query block q0 .. q0 + kBlockQ - 1 visits.
__host__ __device__ inline int qblock_tiles(int q0, int S, int W) {
  const int q_last = q0 + kBlockQ - 1 < S - 1 ? q0 + kBlockQ - 1 : S - 1;
  const int lo = q0 - W + 1 > 0 ? q0 - W + 1 : 0;
  return (q_last - (lo / kTL) * kTL) / kTL + 1;
}
// Query tiles (of kTLdkv) that the key block k0 .. k0 + kBlockK - 1 visits.
__host__ __device__ inline int kblock_tiles(int k0, int S, int W) {
  const int k_last = k0 + kBlockK - 1 < S - 1 ? k0 + kBlockK - 1 : S - 1;
  const int q_end = k_last + W - 1 < S - 1 ? k_last + W - 1 : S - 1;
  return (q_end - k0) / kTLdkv + 1;
}

PB_DEV float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }  // exp2(-inf) = 0

typedef short s16x4 __attribute__((ext_vector_type(4)));
#define PB_LDS __attribute__((address_space(3)))

// ------------------------------------------------------------ LDS tiles
// Every tile is natural: kTL token rows x D features, 2 D bytes per row, the
// 16-byte chunk c of row r stored at chunk c ^ f(r).  For D = 128 (16 chunks
// per row, one 256-byte bank period) f is a 4-bit rotation of r that makes
// both access patterns conflict-free: a 16-byte read by 16 consecutive rows
// at one chunk, and a transposing read of 8 consecutive rows x 4 aligned
// chunks.  D = 64 uses an injective 3-bit variant.  D = 96 (12 chunks, rows
// 192 bytes apart): row r starts at bank group 12 r mod 16 = 4 (3 r mod 4),
// so r mod 4 already spreads rows over the four quarters of the bank period;
// f(r) = (r / 4) mod 4 on the low two chunk bits (which keeps c below 12)
// spreads them within a quarter.  16 rows at one chunk then hit 16 distinct
// bank groups, and so do 4 consecutive rows x 4 aligned chunks.
template <int D>
PB_DEV int rowswz(int r) {
  static_assert(D == 64 || D == 96 || D == 128, "head_dim");
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else if constexpr (D == 96) return (r >> 2) & 3;
  else return ((r & 1) << 2) | ((r >> 1) & 3);
}
template <int D>
PB_DEV int chunk_at(int r, int c) { return c ^ rowswz<D>(r); }

PB_DEV void dma16(const void* g, uint32_t lds_byte_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_byte_addr)
               : "memory", "m0");
}
PB_DEV void dma4(const void* g, uint32_t lds_byte_addr) {  // lane l's 4 bytes -> base + 4 l
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(lds_byte_addr)
               : "memory", "m0");
}
PB_DEV void wait_dma_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// Wait until at most n DMA instructions of this wave are still in flight
// (n uniform; values above 15 wait for all).
PB_DEV void wait_dma_upto(int n) {
#define PB_VMCNT_CASE(k) \
  case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
  switch (n) {
    PB_VMCNT_CASE(1) PB_VMCNT_CASE(2) PB_VMCNT_CASE(3) PB_VMCNT_CASE(4) PB_VMCNT_CASE(5)
    PB_VMCNT_CASE(6) PB_VMCNT_CASE(7) PB_VMCNT_CASE(8) PB_VMCNT_CASE(9) PB_VMCNT_CASE(10)
    PB_VMCNT_CASE(11) PB_VMCNT_CASE(12) PB_VMCNT_CASE(13) PB_VMCNT_CASE(14) PB_VMCNT_CASE(15)
    default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
#undef PB_VMCNT_CASE
}
PB_DEV void block_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// This wave's share of a natural tile, rows row0 .. row0 + kTL - 1 of a
// [rows_valid, ld] token-major matrix, by LDS-DMA (each lane's 16 bytes land
// at the piece's LDS base + 16 * lane).  Rows past rows_valid are read from
// the last valid row: finite values that the window mask always zeroes.
// The tile is cut into 1 KB pieces (one DMA instruction each); with NW
// dividing their number each wave moves a contiguous run, else piece i goes
// to wave i mod NW.  dma_pieces is the number a wave issues.
template <int D, int TL, int NW>
__host__ __device__ constexpr int dma_pieces(int wave) {
  constexpr int NP = TL * 2 * D / 1024;
  return NP % NW == 0 ? NP / NW : (NP - wave + NW - 1) / NW;
}
template <int D, int TL, int NW>
PB_DEV void dma_tile(const bf16* __restrict__ base, int ld, int row0, int rows_valid,
                     uint32_t lds_tile, int wave, int lane) {
  constexpr int RB = 2 * D;
  constexpr int BYTES = TL * RB;
  constexpr int NP = BYTES / 1024;
  static_assert(BYTES % 1024 == 0, "tiles are whole 1 KB pieces");
#pragma unroll
  for (int i = 0; i < (NP + NW - 1) / NW; ++i) {
    const int pc = NP % NW == 0 ? wave * (NP / NW) + i : i * NW + wave;
    if (NP % NW != 0 && pc >= NP) break;  // wave-uniform
    const int piece = pc * 1024;
    const int p = piece + 16 * lane;
    const int row = p / RB, slot = (p / 16) % (RB / 16);
    const int c = chunk_at<D>(row, slot);
    const int t = min(row0 + row, rows_valid - 1);
    dma16(base + (size_t)t * ld + 8 * c, __builtin_amdgcn_readfirstlane(lds_tile + piece));
  }
}

// MFMA operand with 8 consecutive features of token row `row` (k-step ks of
// the feature contraction, lane half h).
template <int D>
PB_DEV bf16x8 frag_row(const unsigned char* tile, int row, int ks, int h) {
  return *reinterpret_cast<const bf16x8*>(tile + row * (2 * D) + chunk_at<D>(row, 2 * ks + h) * 16);
}
// MFMA operand with 8 tokens of feature row `e` of the transposed tile, in
// the order the probabilities sit in a 32 x 32 accumulator: tokens
// 16 s + 4 h + {0..3} then 16 s + 8 + 4 h + {0..3}.  Two transposing reads:
// lane 4 j + q of a 16-lane group addresses token kb + j, features
// (e & ~15) + 4 q .. +3; lane i receives tokens kb .. kb + 3 of feature
// (e & ~15) + i.
template <int D>
PB_DEV bf16x8 frag_tr(const unsigned char* tile, int e, int s, int h, int lane) {
  const int i = lane & 15, j = i >> 2, q = i & 3;
  const int d0 = (e & ~15) + 4 * q;
  const int c = d0 >> 3, off = (d0 & 7) * 2;
  const int t1 = 16 * s + 4 * h + j, t2 = t1 + 8;
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (PB_LDS s16x4*)(tile + t1 * (2 * D) + chunk_at<D>(t1, c) * 16 + off));
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (PB_LDS s16x4*)(tile + t2 * (2 * D) + chunk_at<D>(t2, c) * 16 + off));
  const bf16x4 a4 = __builtin_bit_cast(bf16x4, a), b4 = __builtin_bit_cast(bf16x4, b);
  return bf16x8{a4[0], a4[1], a4[2], a4[3], b4[0], b4[1], b4[2], b4[3]};
}

// Probabilities for MFMA k-step s (16 tokens) from 32-token accumulators.
PB_DEV bf16x8 probs_frag(const f32x16* p, int s) {
  const f32x16& a = p[s >> 1];
  const int o = 8 * (s & 1);
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (bf16)a[o + e];
  return r;
}

PB_DEV f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int e = 0; e < 16; ++e) z[e] = 0.f;
  return z;
}

// 8 consecutive features of one token row from global memory (zero if !ok).
PB_DEV bf16x8 load_row_frag(const bf16* p, bool ok) {
  const u32x4 v = *reinterpret_cast<const u32x4*>(p);
  return ok ? __builtin_bit_cast(bf16x8, v) : bf16x8{};
}

// Work order across heads.  The bf16 kernels' grids are (blocks, heads,
// batch) and workgroups start in linear order, x fastest: head after head.
// Within a head the block index runs from the longest block (most tiles
// under the causal window) to the shortest, so in that order the longest
// blocks of the last heads start only once earlier heads' workgroups have
// left, and the chip idles while they finish.  Renumbering the linear id
// with the block index slowest starts the longest block of every head first.
struct WorkItem {
  int bx, head, b;
};
PB_DEV WorkItem work_item() {
  const int hb_n = (int)(gridDim.y * gridDim.z);
  const int L = (int)(blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z));
  const int hb = L % hb_n;
  return WorkItem{L / hb_n, hb % (int)gridDim.y, hb / (int)gridDim.y};
}

// ====================================================== 16x16x32 tiles
// Tiles for the v_mfma_f32_16x16x32_bf16 kernels, natural token-major like
// the ones above, with their own chunk swizzle: chunk c of row r is stored
// at slot c ^ swz16(r).  The maps are linear in the row bits and were found
// by exhaustive search under a model of the LDS (64 banks of 4 bytes) that
// reproduces the measured behaviour of earlier layouts: a 16-byte read is
// free of conflicts when each 16 lanes hit distinct banks; a transposing
// 8-byte read when each 32 lanes hit distinct banks and, in addition, the
// four rows a 16-lane group reads lie in four distinct 64-byte quarters of
// the bank space (a layout with two of them in one quarter ran the
// forward's O update about six times slower).  Both of the forward's reads
// (K rows in the permuted key order below, one chunk per 16 lanes; the
// transposing reads of V, rows 8 g + j of lane group g) satisfy these for
// head dims 64, 96 and 128; for 96 only the low two chunk bits move, which
// keeps the slot below 12.  Only row bits 0, 1, 3 and 4 enter.
template <int D>
PB_DEV int swz16(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | (((r >> 3) & 1) << 1) | ((r >> 4) & 1);
  else if constexpr (D == 96) return (((r >> 3) & 1) << 1) | ((r >> 4) & 1);
  else return (((r >> 1) & 1) << 2) | (((r >> 3) & 1) << 1) | ((r >> 4) & 1);
}
// The swizzle of tiles read only by transposing reads (V in the forward).
// Same rules, and in addition the two 16-byte halves of a 32-byte row
// segment are never swapped (bit 0 stays), as in the GEMM's transposed
// layout.
template <int D>
PB_DEV int swz16v(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | (((r >> 3) & 1) << 1);
  else if constexpr (D == 96) return ((r >> 3) & 1) << 1;
  else return (((r >> 1) & 1) << 2) | (((r >> 3) & 1) << 1);
}

// Key order inside a 64-key tile for the score MFMAs.  Score block kb (16
// keys; kb = 2 s + h) uses, as its MFMA row i, key 32 s + 8 (i / 4) + 4 h +
// (i mod 4).  The result row i lands in lane group i / 4 as element i mod 4,
// so lane group g holds keys 32 s + 8 g + 0..3 (block 2 s) and + 4..7 (block
// 2 s + 1): exactly the eight consecutive keys that the probability operand
// of the next MFMA (k-step s of 32 keys) wants from that lane group.
PB_DEV int score_key(int kb, int i) { return 32 * (kb >> 1) + 8 * (i >> 2) + 4 * (kb & 1) + (i & 3); }
constexpr int score_row_off(int kb) { return 32 * (kb >> 1) + 4 * (kb & 1); }

// This lane's LDS byte offsets for the forward's fragment reads inside one
// tile.  swz16 depends only on row bits 0, 1, 3 and 4, which are fixed per
// lane for both reads, so each block's row offset (bits 2 and 5) is a
// constant added to one per-lane base: D/32 bases for K and D/16 for V.
//   k[ks]: A operand of K for score block kb, k-step ks (features 32 ks ..
//          + 31) at k[ks] + 2 D score_row_off(kb): lane l supplies row
//          score_key(kb, l & 15), features 32 ks + 8 (l >> 4) .. + 7.
//   v[db]: A operand of V^T for features 16 db .. + 15 and keys 32 s ..
//          + 31, by two transposing reads at v[db] + 2 D (32 s) and
//          + 2 D (32 s + 4): lane 4 j + q of a 16-lane group addresses key
//          base + j, features 16 db + 4 q .. + 3, and receives keys base ..
//          base + 3 of its own feature 16 db + (l & 15); lane group g takes
//          keys 32 s + 8 g .. + 7.
template <int D>
struct FwdLds {
  uint32_t k[D / 32];
  uint32_t v[D / 16];
  PB_DEV explicit FwdLds(int lane) {
    const int i = lane & 15, g = lane >> 4;
    const int rk = score_key(0, i);
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
      k[ks] = (uint32_t)(rk * 2 * D + (((4 * ks + g) ^ swz16<D>(rk)) * 16));
    const int j = i >> 2, q = i & 3;
    const int tv = 8 * g + j;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const int d0 = 16 * db + 4 * q;
      v[db] = (uint32_t)(tv * 2 * D + (((d0 >> 3) ^ swz16v<D>(tv)) * 16) + (d0 & 7) * 2);
    }
  }
};
PB_DEV bf16x8 lds_b128(uint32_t addr) { return *(const PB_LDS bf16x8*)addr; }
// Two transposing reads at addr and addr + gap bytes (four keys each).
PB_DEV bf16x8 lds_tr2(uint32_t addr, uint32_t gap) {
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((PB_LDS s16x4*)addr);
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((PB_LDS s16x4*)(addr + gap));
  const bf16x4 a4 = __builtin_bit_cast(bf16x4, a), b4 = __builtin_bit_cast(bf16x4, b);
  return bf16x8{a4[0], a4[1], a4[2], a4[3], b4[0], b4[1], b4[2], b4[3]};
}
// Values consumed by an empty asm: computed by this point (IR passes would
// otherwise sink them to their first use, out of the phase that interleaves
// them with MFMAs).
PB_DEV void keep(const bf16x8& x) { asm volatile("" ::"v"(__builtin_bit_cast(u32x4, x))); }
PB_DEV void keep(float x) { asm volatile("" ::"v"(x)); }
// Scheduling-group masks (sched_group_barrier): matrix, vector ALU, LDS read.
constexpr int kSgMfma = 0x008, kSgValu = 0x002, kSgDsRead = 0x100;

// LDS-DMA of a TL-row tile in the swz16 layout: this wave's NP / NW 1 KB
// pieces (NP = TL 2 D / 1024, a multiple of NW).  Row r of the tile is token
// row0 + r of a [rows_valid, ld] matrix (rows past the end read the last
// one: finite values the window mask always zeroes).  The lane's 16 bytes
// of piece i are global chunk slot ^ swz(row) of its row (swz16, or swz16v
// with VSWZ); row[i] and cof[i] (that chunk's byte offset) are fixed per
// lane.
template <int D, int TL, int NW, bool VSWZ = false>
struct DmaRows {
  static constexpr int NP = TL * 2 * D / 1024;
  static constexpr int NPW = NP / NW;
  static_assert(NP % NW == 0, "whole pieces per wave");
  int row[NPW];
  uint32_t cof[NPW];
  PB_DEV DmaRows(int wave, int lane) {
    constexpr int RB = 2 * D;
#pragma unroll
    for (int i = 0; i < NPW; ++i) {
      const int p = (wave * NPW + i) * 1024 + 16 * lane;
      row[i] = p / RB;
      const int sw = VSWZ ? swz16v<D>(row[i]) : swz16<D>(row[i]);
      cof[i] = (uint32_t)(((p / 16) % (RB / 16)) ^ sw) * 16u;
    }
  }
  // offsets of this wave's pieces for the tile starting at token row0
  PB_DEV void offsets(int row0, int rows_valid, int ld, uint32_t (&off)[NPW]) const {
#pragma unroll
    for (int i = 0; i < NPW; ++i)
      off[i] = (uint32_t)min(row0 + row[i], rows_valid - 1) * (uint32_t)(2 * ld) + cof[i];
  }
  PB_DEV void issue(const bf16* base, const uint32_t (&off)[NPW], uint32_t lds_tile,
                    int wave) const {
#pragma unroll
    for (int i = 0; i < NPW; ++i)
      dma16s(base, off[i], lds_tile + (uint32_t)((wave * NPW + i) * 1024));
  }
};

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
PB_DEV f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }
PB_DEV f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// Reductions over the four lane groups (lanes l, l ^ 16, l ^ 32, l ^ 48),
// by the two lane-swap instructions.
PB_DEV float max4groups(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false,
                                                  false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
PB_DEV float sum4groups(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false,
                                                  false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
// Sum of the eight bf16 values of an operand, added to acc (two-element dot
// products with (1, 1): the row sums use exactly the rounded probabilities
// that the output MFMA multiplies).
PB_DEV float add_bf16x8(const bf16x8& p, float acc) {
  const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
  acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p[0], p[1]}, one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p[2], p[3]}, one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p[4], p[5]}, one, acc, false);
  return __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p[6], p[7]}, one, acc, false);
}

// ============================================================== forward
// Workgroup: four waves, 128 queries of one (batch row, head); wave w owns
// queries q0 + 32 w .. + 31 as two 16-query column blocks.  Per 64-key tile
// it computes S^T = K Q^T (keys x queries, 4 x 2 blocks of 16 x 16: each
// lane holds 16 scores of each of its two queries), the online softmax, and
// O^T += V^T P^T (D/16 x 2 blocks).  A query's scores of one tile sit in four
// lanes (one per lane group), which share one running maximum: the maximum
// moves, with a cross-lane reduction, only when some lane's scores exceed it
// by more than 8 (base 2), so probabilities stay below 256 and most tiles
// skip both the reduction and the rescale (output and row sum share the
// reference, so the final quotient is unchanged).  Row sums are kept per
// lane and added across the four lanes at the end.
// Software pipeline, so that the matrix cores always have independent work
// next to the vector code: iteration t runs tile t + 1's score MFMAs next to
// tile t's exponentials, then tile t's O^T MFMAs next to tile t + 1's mask
// and maximum.  Each phase (one k-step of the scores, one 16-feature block
// of O^T) is its own scheduling region that reads the next phase's
// fragments while its MFMAs run.  LDS: K in two slots (tile t + 2 loads
// while t + 1 is read), V in three (t + 2 loads while t is read and t + 1
// waits).  Tiles outside a wave's window (one or two at either end of the
// block's range) are masked entirely rather than skipped, which keeps the
// loop free of branches around the pipelined code.
template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void attn_fwd_bf16(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V, int ld,
    bf16* __restrict__ O, int ld_o, float* __restrict__ lse, int S, int H, int W, float scale,
    int cs, int nc, float* __restrict__ po, float* __restrict__ plse) {
  constexpr int TL = kTL;
  constexpr int NB = kBlockQ;
  constexpr int TB = TL * 2 * D;  // bytes per tile
  constexpr int KS = D / 32, DB = D / 16;
  static_assert(kWavesQ == 4 && NB == 128 && TL == 64, "four waves of 32 queries, 64-key tiles");
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(PB_LDS unsigned char*)smem;
  auto k_off = [](int s) { return (uint32_t)(s * TB); };        // K slots 0, 1
  auto v_off = [](int s) { return (uint32_t)((2 + s) * TB); };  // V slots 0, 1, 2

  const int nqb = (S + NB - 1) / NB;
  const WorkItem wi = work_item();
  const int chunk = wi.bx % nc;
  const int q0 = (nqb - 1 - wi.bx / nc) * NB;  // longest rows first
  const int ntot = qblock_tiles(q0, S, W);
  const int t_begin = chunk * cs;
  if (t_begin >= ntot) return;  // this block has fewer chunks than the longest
  const int t_end = min(ntot, t_begin + cs);
  const int n = t_end - t_begin;
  const bool split = ntot > cs;
  const int head = wi.head, b = wi.b;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int g = lane >> 4, col = lane & 15;
  const size_t tok0 = (size_t)b * S;
  const bf16* kb = K + tok0 * ld + head * D;
  const bf16* vb = V + tok0 * ld + head * D;

  const int qw0 = q0 + 32 * wave;
  bf16x8 qf[2][KS];
  {
    const bf16* qb = Q + tok0 * ld + head * D;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int q = qw0 + 16 * j + col;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf[j][ks] = load_row_frag(qb + (size_t)min(q, S - 1) * ld + 32 * ks + 8 * g, q < S);
    }
  }

  const float c2 = scale * kLog2e;
  float m_run[2] = {kNegInf, kNegInf}, l_run[2] = {0.f, 0.f};
  f32x4 o[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db][0] = o[db][1] = zero4();

  const int kv_begin = (max(0, q0 - W + 1) / TL) * TL;
  const DmaRows<D, TL, kWavesQ> dk(wave, lane);
  const DmaRows<D, TL, kWavesQ, true> dv(wave, lane);
  constexpr int PK = DmaRows<D, TL, kWavesQ>::NPW;  // DMA instructions per tile and operand
  const FwdLds<D> la(lane);
  auto issue = [&](int i) {  // tile t_begin + i into K slot i % 2 and V slot i % 3
    uint32_t off[PK];
    dk.offsets(kv_begin + (t_begin + i) * TL, S, ld, off);
    dk.issue(kb, off, lds0 + k_off(i & 1), wave);
    dv.offsets(kv_begin + (t_begin + i) * TL, S, ld, off);
    dv.issue(vb, off, lds0 + v_off(i % 3), wave);
  };

  f32x4 sa[4][2], sb[4][2];  // scores of two consecutive tiles (roles alternate)
  bf16x8 pf[2][2];  // probabilities of tile t [k-step of 32 keys][query block]
  bf16x8 kf[2][4];  // K fragments of two k-steps
  bf16x8 vf[3][2];  // V^T fragments of three feature blocks [block mod 3][k-step]
  float m_use[2];

  auto read_k = [&](uint32_t base, int ks) {
#pragma unroll
    for (int k4 = 0; k4 < 4; ++k4)
      kf[ks & 1][k4] = lds_b128(base + la.k[ks] + 2 * D * score_row_off(k4));
  };
  auto read_v = [&](uint32_t base, int db) {
#pragma unroll
    for (int sp = 0; sp < 2; ++sp)
      vf[db % 3][sp] = lds_tr2(base + la.v[db] + 2 * D * 32 * sp, 2 * D * 4);
  };
  // exponentials of half a probability operand: unit u = (query block
  // u / 4, k-step (u / 2) % 2, half u % 2), four values of block 2 sp + h
  auto exp_unit = [&](const f32x4 (&sc)[4][2], int u) {
    const int j = u >> 2, sp = (u >> 1) & 1, h = u & 1;
    float p[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) p[e] = exp2_hw(fmaf(sc[2 * sp + h][j][e], c2, -m_use[j]));
    const bf16 p0 = (bf16)p[0], p1 = (bf16)p[1], p2 = (bf16)p[2], p3 = (bf16)p[3];
    pf[sp][j][4 * h] = p0, pf[sp][j][4 * h + 1] = p1;
    pf[sp][j][4 * h + 2] = p2, pf[sp][j][4 * h + 3] = p3;
    const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
    l_run[j] = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p0, p1}, one, l_run[j], false);
    l_run[j] = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p2, p3}, one, l_run[j], false);
  };
  // phase ks of the next tile's scores into sn (reads of k-step ks + 1
  // inside), with the current tile's exponential units ks 8 / KS ..
  auto score_phase = [&](uint32_t kbase, int ks, f32x4 (&sn)[4][2]) {
    if (ks + 1 < KS) read_k(kbase, ks + 1);
#pragma unroll
    for (int k4 = 0; k4 < 4; ++k4) {
      sn[k4][0] = mfma16(kf[ks & 1][k4], qf[0][ks], ks ? sn[k4][0] : zero4());
      sn[k4][1] = mfma16(kf[ks & 1][k4], qf[1][ks], ks ? sn[k4][1] : zero4());
    }
  };
  auto score_sched_pattern = [&](int ks, bool valu) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
      if (ks + 1 < KS) __builtin_amdgcn_sched_group_barrier(kSgDsRead, 1, 0);
      if (valu) __builtin_amdgcn_sched_group_barrier(kSgValu, 3, 0);
      __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
      if (valu) __builtin_amdgcn_sched_group_barrier(kSgValu, 3, 0);
    }
  };
  auto score_sched = [&](int ks, bool valu) {
    score_sched_pattern(ks, valu);
    __builtin_amdgcn_sched_barrier(0);
  };
  auto exp_phase = [&](const f32x4 (&sc)[4][2], int ks) {
#pragma unroll
    for (int u = ks * 8 / KS; u < (ks + 1) * 8 / KS; ++u) exp_unit(sc, u);
  };
  auto keep_exps = [&](int ks) {  // the units of exp_phase(ks), done
#pragma unroll
    for (int u = ks * 8 / KS; u < (ks + 1) * 8 / KS; ++u)
      if (u % 2 == 1 || u == (ks + 1) * 8 / KS - 1) keep(pf[(u >> 1) & 1][u >> 2]);
    keep(l_run[0]);
    keep(l_run[1]);
  };
  // mask of a partial tile; its own region
  auto mask_tile = [&](f32x4 (&sc)[4][2], int kv0) {
    const bool full = (kv0 + TL - 1 <= qw0) && (qw0 + 31 - kv0 < W) && (kv0 + TL <= S) &&
                      (qw0 + 32 <= S);
    if (!full) {
#pragma unroll
      for (int k4 = 0; k4 < 4; ++k4)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int key = kv0 + score_key(k4, 4 * g + e);
            const int q = qw0 + 16 * j + col;
            const bool ok = (unsigned)(q - key) < (unsigned)W && key < S;
            sc[k4][j][e] = ok ? sc[k4][j][e] : kNegInf;
          }
    }
  };
  // the scaled lane maxima of a tile's scores
  auto lane_max = [&](const f32x4 (&sc)[4][2], float (&mx)[2]) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float m = sc[0][j][0];
#pragma unroll
      for (int k4 = 0; k4 < 4; ++k4)
#pragma unroll
        for (int e = 0; e < 4; ++e) m = fmaxf(m, sc[k4][j][e]);
      mx[j] = m * c2;
    }
  };
  // phase db of the current tile's O^T update (reads of block db + 2 inside)
  auto pv_phase = [&](uint32_t vbase, int db) {
    if (db + 2 < DB) read_v(vbase, db + 2);
#pragma unroll
    for (int sp = 0; sp < 2; ++sp) {
      o[db][0] = mfma16(vf[db % 3][sp], pf[sp][0], o[db][0]);
      o[db][1] = mfma16(vf[db % 3][sp], pf[sp][1], o[db][1]);
    }
  };
  auto pv_sched_pattern = [&](int db, bool valu) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
      if (db + 2 < DB) __builtin_amdgcn_sched_group_barrier(kSgDsRead, 1, 0);
      if (valu) __builtin_amdgcn_sched_group_barrier(kSgValu, 4, 0);
    }
  };
  // new reference maxima from the lane maxima mx; returns whether any lane
  // rescales, with the factors for O and l
  auto update_max = [&](const float (&mx)[2], float (&alpha)[2]) {
    alpha[0] = alpha[1] = 1.f;
    const bool any = __builtin_amdgcn_ballot_w64(mx[0] > m_run[0] + 8.f || mx[1] > m_run[1] + 8.f);
    if (any) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const float m_new = fmaxf(m_run[j], max4groups(mx[j]));
        alpha[j] = m_new == kNegInf ? 1.f : exp2_hw(m_run[j] - m_new);
        m_run[j] = m_new;
      }
    }
    return any;
  };

  // One iteration: tile i's scores are in cur (masked, m_run covers them).
  // With NEXT, tile i + 1's scores go to nxt next to tile i's exponentials,
  // and its mask and maximum next to tile i's O^T update.
  auto iteration = [&](int i, f32x4 (&cur)[4][2], f32x4 (&nxt)[4][2], auto NEXT) {
    constexpr bool has_next = decltype(NEXT)::value;
#pragma unroll
    for (int j = 0; j < 2; ++j) m_use[j] = m_run[j] == kNegInf ? 0.f : m_run[j];
    wait_dma_upto(has_next ? PK : 0);  // V of tile i and K of tile i + 1 have landed
    block_barrier();  // ... for every wave; the slots of tile i - 1 are free
    if (i + 2 < n) issue(i + 2);
    const uint32_t kbase = lds0 + k_off((i + 1) & 1), vbase = lds0 + v_off(i % 3);
    if (has_next) read_k(kbase, 0);
    read_v(vbase, 0);
    read_v(vbase, 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (has_next) score_phase(kbase, ks, nxt);
      exp_phase(cur, ks);
      score_sched_pattern(ks, true);
      keep_exps(ks);
      __builtin_amdgcn_sched_barrier(0);
    }
    float mx[2] = {kNegInf, kNegInf};
    if (has_next) {
      mask_tile(nxt, kv_begin + (t_begin + i + 1) * TL);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      pv_phase(vbase, db);
      if (has_next && db == 0) lane_max(nxt, mx);
      pv_sched_pattern(db, has_next && db == 0);
      if (has_next && db == 0) keep(mx[0]), keep(mx[1]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (has_next) {
      float alpha[2];
      if (update_max(mx, alpha)) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          l_run[j] *= alpha[j];
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int e = 0; e < 4; ++e) o[db][j][e] *= alpha[j];
        }
      }
    }
  };

  // prologue: tiles 0 and 1 requested; tile 0's scores, mask and maximum
  issue(0);
  if (n > 1) issue(1);
  wait_dma_upto(n > 1 ? 3 * PK : PK);  // K of tile 0
  block_barrier();
  read_k(lds0 + k_off(0), 0);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    score_phase(lds0 + k_off(0), ks, sa);
    score_sched(ks, false);
  }
  {
    mask_tile(sa, kv_begin + t_begin * TL);
    float mx[2], alpha[2];
    lane_max(sa, mx);
    update_max(mx, alpha);  // o and l are zero: nothing to rescale
  }
  using T_ = std::true_type;
  using F_ = std::false_type;
  int i = 0;
  for (; i + 2 < n; i += 2) {
    iteration(i, sa, sb, T_{});
    iteration(i + 1, sb, sa, T_{});
  }
  if (n - i == 2) {
    iteration(i, sa, sb, T_{});
    iteration(i + 1, sb, sa, F_{});
  } else {
    iteration(i, sa, sb, F_{});
  }

#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float l_tot = sum4groups(l_run[j]);
    const int q = qw0 + 16 * j + col;
    if (q >= S) continue;
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    const float mu = m_run[j] == kNegInf ? 0.f : m_run[j];
    const size_t row = ((size_t)b * H + head) * S + q;
    if (!split) {
      bf16* orow = O + (tok0 + q) * ld_o + head * D + 4 * g;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        float v[4] = {o[db][j][0] * inv, o[db][j][1] * inv, o[db][j][2] * inv,
                      o[db][j][3] * inv};
        store4(orow + 16 * db, v);
      }
      if (g == 0) lse[row] = (mu + log2f(l_tot)) * kLn2;
    } else {
      // this chunk's normalised output and its base-2 log-sum-exp (-inf when
      // none of the chunk's keys is visible to the query)
      const size_t bhs = (size_t)gridDim.z * H * S;
      float* prow = po + ((size_t)chunk * bhs + row) * D + 4 * g;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<f32x4*>(prow + 16 * db) =
            f32x4{o[db][j][0] * inv, o[db][j][1] * inv, o[db][j][2] * inv, o[db][j][3] * inv};
      if (g == 0) plse[(size_t)chunk * bhs + row] = l_tot > 0.f ? mu + log2f(l_tot) : kNegInf;
    }
  }
}

// Merge of a split forward: per row, the chunks' normalised outputs weighted
// by 2^(lse_c - lse), lse = log2 sum_c 2^lse_c.  Rows of unsplit blocks are
// left alone (their workgroup wrote the result).  Thread: one row, 8 features.
template <int D>
__global__ __launch_bounds__(256) void attn_fwd_combine(const float* __restrict__ po,
                                                        const float* __restrict__ plse, int cs,
                                                        bf16* __restrict__ O, int ld_o,
                                                        float* __restrict__ lse, int B, int S,
                                                        int H, int W) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t bhs = (size_t)B * H * S;
  const int g = (int)(idx % (D / 8));
  const size_t row = idx / (D / 8);
  if (row >= bhs) return;
  const int t = (int)(row % S);
  const int bh = (int)(row / S), head = bh % H, b = bh / H;
  const int ntot = qblock_tiles((t / kBlockQ) * kBlockQ, S, W);
  if (ntot <= cs) return;
  const int nch = (ntot + cs - 1) / cs;
  float m = kNegInf;
  for (int c = 0; c < nch; ++c) m = fmaxf(m, plse[(size_t)c * bhs + row]);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, l = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float w = exp2_hw(plse[(size_t)c * bhs + row] - m);
    float v[8];
    load8(po + ((size_t)c * bhs + row) * D + 8 * g, v);
    l += w;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = fmaf(w, v[e], acc[e]);
  }
  const float inv = 1.0f / l;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] *= inv;
  store8(O + ((size_t)b * S + t) * ld_o + head * D + 8 * g, acc);
  if (g == 0) lse[row] = (m + log2f(l)) * kLn2;
}

// Merge of a split dQ or dK/dV: the chunks' fp32 partial sums added in chunk
// order (KEYS: rows are key blocks, else query blocks).  p2 / o2 may be NULL.
template <int D, bool KEYS>
__global__ __launch_bounds__(256) void attn_sum_combine(const float* __restrict__ p1,
                                                        const float* __restrict__ p2, int cs,
                                                        bf16* __restrict__ o1,
                                                        bf16* __restrict__ o2, int ld, int B,
                                                        int S, int H, int W) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t bhs = (size_t)B * H * S;
  const int g = (int)(idx % (D / 8));
  const size_t row = idx / (D / 8);
  if (row >= bhs) return;
  const int t = (int)(row % S);
  const int bh = (int)(row / S), head = bh % H, b = bh / H;
  const int nb = KEYS ? kBlockK : kBlockQ;
  const int ntot = KEYS ? kblock_tiles((t / nb) * nb, S, W) : qblock_tiles((t / nb) * nb, S, W);
  if (ntot <= cs) return;
  const int nch = (ntot + cs - 1) / cs;
  const size_t out = ((size_t)b * S + t) * ld + head * D + 8 * g;
  for (int which = 0; which < 2; ++which) {
    const float* p = which ? p2 : p1;
    bf16* o = which ? o2 : o1;
    if (!p) break;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < nch; ++c) {
      float v[8];
      load8(p + ((size_t)c * bhs + row) * D + 8 * g, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += v[e];
    }
    store8(o + out, acc);
  }
}

// ===================================================== backward: delta
template <typename T>
__global__ __launch_bounds__(256) void attn_delta_kernel(const T* __restrict__ O, int ld_o,
                                                         const T* __restrict__ dO, int ld_do,
                                                         float* __restrict__ delta, int B, int S,
                                                         int H, int D) {
  const int idx = blockIdx.x * 256 + threadIdx.x;  // (b, t, head)
  if (idx >= B * S * H) return;
  const int head = idx % H, bt = idx / H;
  const int b = bt / S, t = bt % S;
  const T* o = O + (size_t)bt * ld_o + head * D;
  const T* g = dO + (size_t)bt * ld_do + head * D;
  float acc = 0.f;
  for (int e = 0; e < D; e += 8) {
    float a[8], c[8];
    load8(o + e, a);
    load8(g + e, c);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += a[i] * c[i];
  }
  delta[((size_t)b * H + head) * S + t] = acc;
}

// ====================================================== backward: dK, dV
// Workgroup: 64 keys in two groups of 32, four waves.  Per key group, wave
// "P" computes S = Q K^T and P = exp(S - lse), hands P to its partner through
// LDS, and accumulates dV^T += dO^T P; wave "dS" computes dP = dO V^T, forms
// dS = P (dP - delta) and accumulates dK^T += Q^T dS.  Each wave so holds one
// operand fragment set (K or V of its 32 keys) and one accumulator block
// instead of two, and both roles run the same matrix code on different
// tiles: half the registers of one wave doing both, and no repeated work.
// The transposed operands are read from the natural Q and dO tiles.
template <int D>
PB_DEV void dkdv_body(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V, int ld,
    const bf16* __restrict__ dO, int ld_o, const float* __restrict__ lse,
    const float* __restrict__ delta, bf16* __restrict__ dK, bf16* __restrict__ dV, int ld_d,
    int S, int H, int W, float scale, int cs, int nc, float* __restrict__ pdk,
    float* __restrict__ pdv, int bx, int head, int b) {
  constexpr int TL = kTLdkv;
  constexpr int NB = kBlockK;
  constexpr int TB = TL * 2 * D;
  constexpr int STAGE = 2 * TB + 2 * TL * 4;  // Q, dO, then lse and delta rows
  constexpr int PBUF = 64 * 16 * 4;           // one wave's P: 16 fp32 per lane
  constexpr int NS = kStagesDkdv;             // tiles in flight: loads run NS - 1 ahead
  static_assert(TL == 32 && NB == 64 && kWavesK == 4, "two key groups x two roles");
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(PB_LDS unsigned char*)smem;
  auto q_off = [&](int s) { return s * STAGE; };
  auto g_off = [&](int s) { return s * STAGE + TB; };
  auto l_off = [&](int s) { return s * STAGE + 2 * TB; };

  const int chunk = bx % nc;
  const int k0 = (bx / nc) * NB;
  const int ntot = kblock_tiles(k0, S, W);
  const int t_begin = chunk * cs;
  if (t_begin >= ntot) return;  // this block has fewer chunks than the longest
  const int t_end = min(ntot, t_begin + cs);
  const bool split = ntot > cs;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int grp = wave & 1;
  const bool pside = wave < 2;
  const int fr = lane & 31, fh = lane >> 5;
  const size_t tok0 = (size_t)b * S;
  const bf16* qb = Q + tok0 * ld + head * D;
  const bf16* gb = dO + tok0 * ld_o + head * D;
  const float* lseb = lse + ((size_t)b * H + head) * S;
  const float* delb = delta + ((size_t)b * H + head) * S;
  float* pbuf = (float*)(smem + NS * STAGE + grp * PBUF);

  const int kw0 = k0 + 32 * grp;
  const int key = kw0 + fr;
  // K (P side) or V (dS side) rows of this wave's 32 keys
  const bf16* kvb = (pside ? K : V) + tok0 * ld + head * D;
  bf16x8 kvf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    kvf[ks] = load_row_frag(kvb + (size_t)min(key, S - 1) * ld + 16 * ks + 8 * fh, key < S);
  f32x16 acc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc[i] = zero16();

  const float c2 = scale * kLog2e;

  // Stage of the i-th tile of this chunk: Q and dO tiles, and the tile's 32
  // lse and 32 delta values (one 4-byte DMA by wave 0; rows past the end are
  // read from the last row: finite values that the mask always zeroes).
  // DMA instructions per wave per stage: dma_tile moves 1 KB pieces.
  const int per_stage = 2 * dma_pieces<D, TL, kWavesK>(wave) + (wave == 0 ? 1 : 0);
  const int nt = t_end - t_begin;
  auto issue_stage = [&](int i) {
    const int s = i % NS;
    const int qs = k0 + (t_begin + i) * TL;
    dma_tile<D, TL, kWavesK>(qb, ld, qs, S, lds0 + q_off(s), wave, lane);
    dma_tile<D, TL, kWavesK>(gb, ld_o, qs, S, lds0 + g_off(s), wave, lane);
    if (wave == 0) {
      const int r = min(qs + (lane & 31), S - 1);
      dma4((lane < 32 ? lseb : delb) + r, __builtin_amdgcn_readfirstlane(lds0 + l_off(s)));
    }
  };
#pragma unroll
  for (int i = 0; i < NS - 1; ++i)
    if (i < nt) issue_stage(i);

  for (int i = 0; i < nt; ++i) {
    const int t = t_begin + i;
    const int cur = i % NS;
    const int qs = k0 + t * TL;
    // stage i has landed once at most the newer stages' loads are in flight
    wait_dma_upto(min(nt - 1 - i, NS - 2) * per_stage);
    block_barrier();  // ... for every wave; and every wave is done with tile i - 1
    if (i + NS - 1 < nt) issue_stage(i + NS - 1);
    const unsigned char* qt = smem + q_off(cur);
    const unsigned char* gt = smem + g_off(cur);
    const float* ls = (const float*)(smem + l_off(cur));
    // Every tile runs unconditionally: where none of a key group's pairs is
    // inside the window the mask zeroes P, hence dS, and the sums stay exact.
    // Lane holds key `key` and queries qs + 8 j + 4 fh + i of element 4 j + i.
    f32x16 sc = zero16();  // S (P side) or dP (dS side)
    const unsigned char* nt = pside ? qt : gt;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_row<D>(nt, fr, ks, fh), kvf[ks], sc, 0,
                                                   0, 0);
    if (pside) {
      const bool full = (qs >= kw0 + 31) && (qs + TL - 1 - kw0 < W) && (qs + TL <= S) &&
                        (kw0 + 32 <= S);
      if (!full) {
        const int d0 = qs + 4 * fh - key, s0 = S - qs - 4 * fh;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int c = 8 * (r >> 2) + (r & 3);
          const bool ok = (unsigned)(d0 + c) < (unsigned)W && c < s0;
          sc[r] = ok ? sc[r] : kNegInf;
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 L4 = *reinterpret_cast<const f32x4*>(ls + 8 * j + 4 * fh);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          sc[4 * j + i] = exp2_hw(fmaf(sc[4 * j + i], c2, -L4[i] * kLog2e));
        *reinterpret_cast<f32x4*>(pbuf + (j * 64 + lane) * 4) =
            f32x4{sc[4 * j], sc[4 * j + 1], sc[4 * j + 2], sc[4 * j + 3]};
      }
    }
    block_barrier();  // P of this tile is visible to the dS side
    if (!pside) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 P4 = *reinterpret_cast<const f32x4*>(pbuf + (j * 64 + lane) * 4);
        const f32x4 D4 = *reinterpret_cast<const f32x4*>(ls + TL + 8 * j + 4 * fh);
#pragma unroll
        for (int i = 0; i < 4; ++i) sc[4 * j + i] = P4[i] * (sc[4 * j + i] - D4[i]);
      }
    }
    const unsigned char* tt = pside ? gt : qt;  // dO^T with P, Q^T with dS
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int s2 = 0; s2 < TL / 16; ++s2)
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            frag_tr<D>(tt, 32 * db + fr, s2, fh, lane), probs_frag(&sc, s2), acc[db], 0, 0, 0);
  }

  if (key < S) {
    const float mul = pside ? 1.f : scale;  // dV, or dK with the score scale
    if (split) {
      const size_t bhs = (size_t)gridDim.z * H * S;
      float* prow =
          (pside ? pdv : pdk) + ((size_t)chunk * bhs + ((size_t)b * H + head) * S + key) * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<f32x4*>(prow + 32 * db + 8 * j + 4 * fh) =
              f32x4{acc[db][4 * j] * mul, acc[db][4 * j + 1] * mul, acc[db][4 * j + 2] * mul,
                    acc[db][4 * j + 3] * mul};
    } else {
      bf16* orow = (pside ? dV : dK) + (tok0 + key) * ld_d + head * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float a[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) a[i] = acc[db][4 * j + i] * mul;
          store4(orow + 32 * db + 8 * j + 4 * fh, a);
        }
    }
  }
}

// ============================================================ backward: dQ
// Workgroup: 32 kWavesQ queries; per key tile: S^T = K Q^T and dP^T = V dO^T,
// dS^T = P^T (dP^T - delta), dQ^T += K^T dS^T (K^T read from the natural K
// tile).
template <int D>
PB_DEV void dq_body(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V, int ld,
    const bf16* __restrict__ dO, int ld_o, const float* __restrict__ lse,
    const float* __restrict__ delta, bf16* __restrict__ dQ, int ld_d, int S, int H, int W,
    float scale, int cs, int nc, float* __restrict__ pdq, int bx, int head, int b) {
  constexpr int TL = kTL;
  constexpr int NB = kBlockQ;
  constexpr int TB = TL * 2 * D;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(PB_LDS unsigned char*)smem;
  auto k_off = [&](int s) { return (2 * s) * TB; };
  auto v_off = [&](int s) { return (2 * s + 1) * TB; };

  const int nqb = (S + NB - 1) / NB;
  const int chunk = bx % nc;
  const int q0 = (nqb - 1 - bx / nc) * NB;
  const int ntot = qblock_tiles(q0, S, W);
  const int t_begin = chunk * cs;
  if (t_begin >= ntot) return;  // this block has fewer chunks than the longest
  const int t_end = min(ntot, t_begin + cs);
  const bool split = ntot > cs;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int fr = lane & 31, fh = lane >> 5;
  const size_t tok0 = (size_t)b * S;
  const bf16* qb = Q + tok0 * ld + head * D;
  const bf16* kb = K + tok0 * ld + head * D;
  const bf16* vb = V + tok0 * ld + head * D;
  const bf16* gb = dO + tok0 * ld_o + head * D;

  const int qw0 = q0 + 32 * wave;
  const int q = qw0 + fr;
  const int qc = min(q, S - 1);
  bf16x8 qf[D / 16], gf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    qf[ks] = load_row_frag(qb + (size_t)qc * ld + 16 * ks + 8 * fh, q < S);
    gf[ks] = load_row_frag(gb + (size_t)qc * ld_o + 16 * ks + 8 * fh, q < S);
  }
  const size_t row_off = ((size_t)b * H + head) * S;
  const float L2 = q < S ? lse[row_off + q] * kLog2e : 0.f;
  const float Dq = q < S ? delta[row_off + q] : 0.f;
  const float c2 = scale * kLog2e;

  f32x16 dq[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) dq[i] = zero16();

  const int kv_begin = (max(0, q0 - W + 1) / TL) * TL;
  const int w_lo = qw0 - W + 1, w_hi = min(qw0 + 31, S - 1);

  dma_tile<D, TL, kWavesQ>(kb, ld, kv_begin + t_begin * TL, S, lds0 + k_off(0), wave, lane);
  dma_tile<D, TL, kWavesQ>(vb, ld, kv_begin + t_begin * TL, S, lds0 + v_off(0), wave, lane);

  for (int t = t_begin; t < t_end; ++t) {
    const int cur = (t - t_begin) & 1;
    const int kv0 = kv_begin + t * TL;
    wait_dma_all();
    block_barrier();
    if (t + 1 < t_end) {
      dma_tile<D, TL, kWavesQ>(kb, ld, kv0 + TL, S, lds0 + k_off(cur ^ 1), wave, lane);
      dma_tile<D, TL, kWavesQ>(vb, ld, kv0 + TL, S, lds0 + v_off(cur ^ 1), wave, lane);
    }
    if (qw0 < S && kv0 <= w_hi && kv0 + TL - 1 >= w_lo) {
      const unsigned char* kt = smem + k_off(cur);
      const unsigned char* vt = smem + v_off(cur);
      f32x16 p[TL / 32], ds[TL / 32];
#pragma unroll
      for (int h2 = 0; h2 < TL / 32; ++h2) {
        p[h2] = zero16();
        ds[h2] = zero16();
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          p[h2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_row<D>(kt, 32 * h2 + fr, ks, fh),
                                                          qf[ks], p[h2], 0, 0, 0);
          ds[h2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_row<D>(vt, 32 * h2 + fr, ks, fh),
                                                           gf[ks], ds[h2], 0, 0, 0);
        }
      }
      const bool full = (kv0 + TL - 1 <= qw0) && (qw0 + 31 - kv0 < W) && (kv0 + TL <= S) &&
                        (qw0 + 32 <= S);
      if (!full) {
        const int d0 = q - kv0 - 4 * fh, s0 = S - kv0 - 4 * fh;
#pragma unroll
        for (int h2 = 0; h2 < TL / 32; ++h2)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int c = 32 * h2 + 8 * (r >> 2) + (r & 3);
            const bool ok = (unsigned)(d0 - c) < (unsigned)W && c < s0;
            p[h2][r] = ok ? p[h2][r] : kNegInf;
          }
      }
#pragma unroll
      for (int h2 = 0; h2 < TL / 32; ++h2)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          ds[h2][r] = exp2_hw(fmaf(p[h2][r], c2, -L2)) * (ds[h2][r] - Dq);
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int s2 = 0; s2 < TL / 16; ++s2)
          dq[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              frag_tr<D>(kt, 32 * db + fr, s2, fh, lane), probs_frag(ds, s2), dq[db], 0, 0, 0);
    }
  }

  if (q < S && split) {
    const size_t bhs = (size_t)gridDim.z * H * S;
    float* prow = pdq + ((size_t)chunk * bhs + row_off + q) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<f32x4*>(prow + 32 * db + 8 * j + 4 * fh) =
            f32x4{dq[db][4 * j] * scale, dq[db][4 * j + 1] * scale, dq[db][4 * j + 2] * scale,
                  dq[db][4 * j + 3] * scale};
  } else if (q < S) {
    bf16* dqr = dQ + (tok0 + q) * ld_d + head * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float a[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = dq[db][4 * j + i] * scale;
        store4(dqr + 32 * db + 8 * j + 4 * fh, a);
      }
  }
}

// Both backward kernels in one launch: workgroups 0 .. nxk - 1 of the x grid
// are dK/dV blocks, the rest dQ blocks.  They are independent given delta;
// sharing a launch lets the short dQ blocks fill the CUs that the dK/dV
// blocks leave idle (both grids alone are too small for the chip at few
// heads), instead of running one after the other.
template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void attn_bwd_bf16(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V, int ld,
    const bf16* __restrict__ dO, int ld_o, const float* __restrict__ lse,
    const float* __restrict__ delta, bf16* __restrict__ dQ, bf16* __restrict__ dK,
    bf16* __restrict__ dV, int ld_d, int S, int H, int W, float scale, int kv_cs, int kv_nc,
    int nxk, int q_cs, int q_nc, float* __restrict__ pdk, float* __restrict__ pdv,
    float* __restrict__ pdq) {
  static_assert(64 * kWavesK == 256 && 64 * kWavesQ == 256, "one block size for both roles");
  // rank r of the work order (block index slowest, see work_item) alternates
  // the two roles, each longest first, until the shorter list runs out
  const WorkItem wi = work_item();
  const int r = wi.bx, nxq = (int)gridDim.x - nxk, mn = min(nxk, nxq);
  int bx;  // < nxk: dK/dV block bx; else dQ block bx - nxk
  if (r < 2 * mn) bx = (r & 1) ? nxk + (r >> 1) : (r >> 1);
  else bx = nxk > nxq ? r - mn : nxk + (r - mn);
  if (bx < nxk)
    dkdv_body<D>(Q, K, V, ld, dO, ld_o, lse, delta, dK, dV, ld_d, S, H, W, scale, kv_cs, kv_nc,
                 pdk, pdv, bx, wi.head, wi.b);
  else
    dq_body<D>(Q, K, V, ld, dO, ld_o, lse, delta, dQ, ld_d, S, H, W, scale, q_cs, q_nc, pdq,
               bx - nxk, wi.head, wi.b);
}

// ============================================================ fp32 path
template <int D>
__global__ __launch_bounds__(64) void attn_fwd_f32(const float* __restrict__ Q,
                                                   const float* __restrict__ K,
                                                   const float* __restrict__ V, int ld,
                                                   float* __restrict__ O, int ld_o,
                                                   float* __restrict__ lse, int S, int H, int W,
                                                   float scale) {
  const int q = blockIdx.x * 64 + threadIdx.x, head = blockIdx.y, b = blockIdx.z;
  if (q >= S) return;
  const size_t tok0 = (size_t)b * S;
  const float* qr = Q + (tok0 + q) * ld + head * D;
  float qv[D], acc[D];
  for (int e = 0; e < D; ++e) { qv[e] = qr[e]; acc[e] = 0.f; }
  float m = kNegInf, l = 0.f;
  for (int j = max(0, q - W + 1); j <= q; ++j) {
    const float* kr = K + (tok0 + j) * ld + head * D;
    const float* vr = V + (tok0 + j) * ld + head * D;
    float s = 0.f;
    for (int e = 0; e < D; ++e) s = fmaf(qv[e], kr[e], s);
    s *= scale;
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn), p = expf(s - mn);
    l = l * a + p;
    for (int e = 0; e < D; ++e) acc[e] = acc[e] * a + p * vr[e];
    m = mn;
  }
  float* orow = O + (tok0 + q) * ld_o + head * D;
  for (int e = 0; e < D; ++e) orow[e] = acc[e] / l;
  lse[((size_t)b * H + head) * S + q] = m + logf(l);
}

template <int D>
__global__ __launch_bounds__(64) void attn_dq_f32(const float* __restrict__ Q,
                                                  const float* __restrict__ K,
                                                  const float* __restrict__ V, int ld,
                                                  const float* __restrict__ dO, int ld_o,
                                                  const float* __restrict__ lse,
                                                  const float* __restrict__ delta,
                                                  float* __restrict__ dQ, int ld_d, int S, int H,
                                                  int W, float scale) {
  const int q = blockIdx.x * 64 + threadIdx.x, head = blockIdx.y, b = blockIdx.z;
  if (q >= S) return;
  const size_t tok0 = (size_t)b * S;
  const float* qr = Q + (tok0 + q) * ld + head * D;
  const float* gr = dO + (tok0 + q) * ld_o + head * D;
  float qv[D], gv[D], acc[D];
  for (int e = 0; e < D; ++e) { qv[e] = qr[e]; gv[e] = gr[e]; acc[e] = 0.f; }
  const size_t ro = ((size_t)b * H + head) * S + q;
  const float L = lse[ro], Dq = delta[ro];
  for (int j = max(0, q - W + 1); j <= q; ++j) {
    const float* kr = K + (tok0 + j) * ld + head * D;
    const float* vr = V + (tok0 + j) * ld + head * D;
    float s = 0.f, dp = 0.f;
    for (int e = 0; e < D; ++e) {
      s = fmaf(qv[e], kr[e], s);
      dp = fmaf(gv[e], vr[e], dp);
    }
    const float ds = expf(s * scale - L) * (dp - Dq);
    for (int e = 0; e < D; ++e) acc[e] = fmaf(ds, kr[e], acc[e]);
  }
  float* out = dQ + (tok0 + q) * ld_d + head * D;
  for (int e = 0; e < D; ++e) out[e] = acc[e] * scale;
}

template <int D>
__global__ __launch_bounds__(64) void attn_dkdv_f32(const float* __restrict__ Q,
                                                    const float* __restrict__ K,
                                                    const float* __restrict__ V, int ld,
                                                    const float* __restrict__ dO, int ld_o,
                                                    const float* __restrict__ lse,
                                                    const float* __restrict__ delta,
                                                    float* __restrict__ dK, float* __restrict__ dV,
                                                    int ld_d, int S, int H, int W, float scale) {
  const int j = blockIdx.x * 64 + threadIdx.x, head = blockIdx.y, b = blockIdx.z;
  if (j >= S) return;
  const size_t tok0 = (size_t)b * S;
  const float* kr = K + (tok0 + j) * ld + head * D;
  const float* vr = V + (tok0 + j) * ld + head * D;
  float kv[D], vv[D], dk[D], dv[D];
  for (int e = 0; e < D; ++e) { kv[e] = kr[e]; vv[e] = vr[e]; dk[e] = 0.f; dv[e] = 0.f; }
  const size_t ro = ((size_t)b * H + head) * S;
  const int i_end = min(S - 1, j + W - 1);
  for (int i = j; i <= i_end; ++i) {
    const float* qr = Q + (tok0 + i) * ld + head * D;
    const float* gr = dO + (tok0 + i) * ld_o + head * D;
    float s = 0.f, dp = 0.f;
    for (int e = 0; e < D; ++e) {
      s = fmaf(qr[e], kv[e], s);
      dp = fmaf(gr[e], vv[e], dp);
    }
    const float p = expf(s * scale - lse[ro + i]);
    const float ds = p * (dp - delta[ro + i]);
    for (int e = 0; e < D; ++e) {
      dv[e] = fmaf(p, gr[e], dv[e]);
      dk[e] = fmaf(ds, qr[e], dk[e]);
    }
  }
  float* dko = dK + (tok0 + j) * ld_d + head * D;
  float* dvo = dV + (tok0 + j) * ld_d + head * D;
  for (int e = 0; e < D; ++e) {
    dko[e] = dk[e] * scale;
    dvo[e] = dv[e];
  }
}

template <int D>
size_t fwd_lds() { return 5 * (size_t)kTL * 2 * D; }  // K: two slots, V: three
template <int D>
size_t dkdv_lds() {
  return kStagesDkdv * (2 * (size_t)kTLdkv * 2 * D + 2 * kTLdkv * 4) + 2 * 64 * 16 * 4;
}
template <int D>
size_t dq_lds() { return 2 * 2 * (size_t)kTL * 2 * D; }

size_t part_floats(const AttnShape& a, int n) {
  return n > 1 ? (size_t)n * a.batch * a.heads * a.seq * a.head_dim : 0;
}
size_t lse_floats(const AttnShape& a, int n) {
  return n > 1 ? (size_t)n * a.batch * a.heads * a.seq : 0;
}
size_t round256(size_t v) { return (v + 255) & ~(size_t)255; }
unsigned combine_grid(const AttnShape& a) {
  return (unsigned)(((size_t)a.batch * a.heads * a.seq * (a.head_dim / 8) + 255) / 256);
}

template <int D>
void fwd_d(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v, int ld,
           void* o, int ld_o, float* lse, void* part, size_t part_bytes, hipStream_t s) {
  const float scale = 1.0f / sqrtf((float)D);
  if (dt == Dt::BF16) {
    AttnSplit p = attn_split_plan(dt, a);
    if (!part || part_bytes < attn_fwd_partial_bytes(a, p)) p.fwd_chunk = kUnsplit, p.fwd_n = 1;
    float* po = (float*)part;
    float* plse = po ? (float*)((char*)part + round256(part_floats(a, p.fwd_n) * 4)) : nullptr;
    dim3 g((a.seq + kBlockQ - 1) / kBlockQ * p.fwd_n, a.heads, a.batch);
    attn_fwd_bf16<D><<<g, 64 * kWavesQ, fwd_lds<D>(), s>>>(
        (const bf16*)q, (const bf16*)k, (const bf16*)v, ld, (bf16*)o, ld_o, lse, a.seq, a.heads,
        a.window, scale, p.fwd_chunk, p.fwd_n, po, plse);
    if (p.fwd_n > 1)
      attn_fwd_combine<D><<<combine_grid(a), 256, 0, s>>>(po, plse, p.fwd_chunk, (bf16*)o, ld_o,
                                                          lse, a.batch, a.seq, a.heads, a.window);
  } else {
    dim3 g((a.seq + 63) / 64, a.heads, a.batch);
    attn_fwd_f32<D><<<g, 64, 0, s>>>((const float*)q, (const float*)k, (const float*)v, ld,
                                     (float*)o, ld_o, lse, a.seq, a.heads, a.window, scale);
  }
}

template <int D>
void bwd_d(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v, int ld,
           const void* o, int ld_o, const void* d_o, int ld_do, const float* lse, float* delta,
           bool delta_ready, void* dq, void* dk, void* dv, int ld_d, void* part,
           size_t part_bytes, hipStream_t s) {
  const float scale = 1.0f / sqrtf((float)D);
  const int nrows = a.batch * a.seq * a.heads;
  if (dt == Dt::BF16) {
    if (!delta_ready)
      attn_delta_kernel<bf16><<<(nrows + 255) / 256, 256, 0, s>>>(
          (const bf16*)o, ld_o, (const bf16*)d_o, ld_do, delta, a.batch, a.seq, a.heads, D);
    AttnSplit p = attn_bwd_split_plan(dt, a);
    if (!part || part_bytes < attn_bwd_partial_bytes(a, p)) {
      p.fwd_chunk = p.kv_chunk = kUnsplit;
      p.fwd_n = p.kv_n = 1;
    }
    // dK, dV and dQ partials side by side (the two roles run concurrently)
    float* pdk = (float*)part;
    float* pdv = pdk ? pdk + part_floats(a, p.kv_n) : nullptr;
    float* pdq = pdk ? pdv + part_floats(a, p.kv_n) : nullptr;
    const int nxk = (a.seq + kBlockK - 1) / kBlockK * p.kv_n;
    const int nxq = (a.seq + kBlockQ - 1) / kBlockQ * p.fwd_n;
    dim3 g(nxk + nxq, a.heads, a.batch);
    attn_bwd_bf16<D><<<g, 256, std::max(dkdv_lds<D>(), dq_lds<D>()), s>>>(
        (const bf16*)q, (const bf16*)k, (const bf16*)v, ld, (const bf16*)d_o, ld_do, lse, delta,
        (bf16*)dq, (bf16*)dk, (bf16*)dv, ld_d, a.seq, a.heads, a.window, scale, p.kv_chunk,
        p.kv_n, nxk, p.fwd_chunk, p.fwd_n, pdk, pdv, pdq);
    if (p.kv_n > 1)
      attn_sum_combine<D, true><<<combine_grid(a), 256, 0, s>>>(
          pdk, pdv, p.kv_chunk, (bf16*)dk, (bf16*)dv, ld_d, a.batch, a.seq, a.heads, a.window);
    if (p.fwd_n > 1)
      attn_sum_combine<D, false><<<combine_grid(a), 256, 0, s>>>(
          pdq, nullptr, p.fwd_chunk, (bf16*)dq, nullptr, ld_d, a.batch, a.seq, a.heads,
          a.window);
  } else {
    if (!delta_ready)
      attn_delta_kernel<float><<<(nrows + 255) / 256, 256, 0, s>>>(
        (const float*)o, ld_o, (const float*)d_o, ld_do, delta, a.batch, a.seq, a.heads, D);
    dim3 g((a.seq + 63) / 64, a.heads, a.batch);
    attn_dq_f32<D><<<g, 64, 0, s>>>((const float*)q, (const float*)k, (const float*)v, ld,
                                    (const float*)d_o, ld_do, lse, delta, (float*)dq, ld_d,
                                    a.seq, a.heads, a.window, scale);
    attn_dkdv_f32<D><<<g, 64, 0, s>>>((const float*)q, (const float*)k, (const float*)v, ld,
                                      (const float*)d_o, ld_do, lse, delta, (float*)dk,
                                      (float*)dv, ld_d, a.seq, a.heads, a.window, scale);
  }
}

}  // namespace

// Split only when a kernel's grid has fewer than kSplitBelow waves; then aim
// for about kSplitTarget waves, with chunks of at least two tiles.  With the
// longest blocks of every head started first (work_item), the split only has
// to shorten the longest blocks: at the 175B share (192 forward blocks) two
// chunks per block run the forward in 0.042 ms, four in 0.045, none 0.054.
constexpr long long kSplitBelow = 2048;
constexpr long long kSplitTarget = 1536;

AttnSplit attn_split_plan(Dt dt, const AttnShape& a) {
  AttnSplit p{kUnsplit, 1, kUnsplit, 1};
  if (dt != Dt::BF16) return p;
  auto choose = [&](int block, int waves, bool keys, int& chunk, int& n) {
    const int nb = (a.seq + block - 1) / block;
    const long long w = (long long)nb * a.heads * a.batch * waves;
    if (w >= kSplitBelow) return;
    int max_tiles = 1;
    for (int i = 0; i < nb; ++i)
      max_tiles = std::max(max_tiles, keys ? kblock_tiles(i * block, a.seq, a.window)
                                           : qblock_tiles(i * block, a.seq, a.window));
    const int want = (int)((kSplitTarget + w - 1) / w);
    const int m = std::min(want, (max_tiles + 1) / 2);
    if (m < 2) return;
    chunk = (max_tiles + m - 1) / m;
    n = (max_tiles + chunk - 1) / chunk;
    if (n < 2) chunk = kUnsplit, n = 1;
  };
  choose(kBlockQ, kWavesQ, false, p.fwd_chunk, p.fwd_n);
  choose(kBlockK, kWavesK, true, p.kv_chunk, p.kv_n);
  return p;
}

AttnSplit attn_bwd_split_plan(Dt dt, const AttnShape& a) {
  AttnSplit p = attn_split_plan(dt, a);
  // both roles share one launch: split only when together they are too few
  const long long blocks = (long long)((a.seq + kBlockK - 1) / kBlockK +
                                       (a.seq + kBlockQ - 1) / kBlockQ) * a.heads * a.batch;
  if (blocks * kWavesK >= kSplitBelow) p = AttnSplit{kUnsplit, 1, kUnsplit, 1};
  return p;
}

size_t attn_fwd_partial_bytes(const AttnShape& a, const AttnSplit& p) {
  if (p.fwd_n < 2) return 0;
  return round256(part_floats(a, p.fwd_n) * 4) + round256(lse_floats(a, p.fwd_n) * 4);
}

size_t attn_bwd_partial_bytes(const AttnShape& a, const AttnSplit& p) {
  return (2 * part_floats(a, p.kv_n) + part_floats(a, p.fwd_n)) * 4;
}

void launch_attn_forward(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v,
                         int ld_qkv, void* o, int ld_o, float* lse, void* part,
                         size_t part_bytes, hipStream_t s) {
  if (a.head_dim == 64) fwd_d<64>(dt, a, q, k, v, ld_qkv, o, ld_o, lse, part, part_bytes, s);
  else if (a.head_dim == 96) fwd_d<96>(dt, a, q, k, v, ld_qkv, o, ld_o, lse, part, part_bytes, s);
  else fwd_d<128>(dt, a, q, k, v, ld_qkv, o, ld_o, lse, part, part_bytes, s);
}

void launch_attn_backward(Dt dt, const AttnShape& a, const void* q, const void* k, const void* v,
                          int ld_qkv, const void* o, int ld_o, const void* d_o, int ld_do,
                          const float* lse, float* delta, bool delta_ready, void* dq, void* dk,
                          void* dv, int ld_d, void* part, size_t part_bytes, hipStream_t s) {
  if (a.head_dim == 64)
    bwd_d<64>(dt, a, q, k, v, ld_qkv, o, ld_o, d_o, ld_do, lse, delta, delta_ready, dq, dk, dv,
              ld_d, part, part_bytes, s);
  else if (a.head_dim == 96)
    bwd_d<96>(dt, a, q, k, v, ld_qkv, o, ld_o, d_o, ld_do, lse, delta, delta_ready, dq, dk, dv,
              ld_d, part, part_bytes, s);
  else
    bwd_d<128>(dt, a, q, k, v, ld_qkv, o, ld_o, d_o, ld_do, lse, delta, delta_ready, dq, dk, dv,
              ld_d, part, part_bytes, s);
}

}  // namespace pb
