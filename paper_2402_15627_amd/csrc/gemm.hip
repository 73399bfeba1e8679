// Projection GEMMs of the parallel block with fused epilogues.
//
// bf16 path: 256x256 output tile per workgroup of eight waves (each wave
// 64x128).  Two kernels share the tile, the wave layout and the epilogues:
//   - K a multiple of 64 (every GEMM of the block at the benchmarked sizes):
//     MFMA v_mfma_f32_16x16x32_bf16, operands reach LDS by LDS-DMA, K-tiles
//     of 64 through two stages, fragments read two phases ahead and the
//     barrier placed before the K-tile's last two phases (see the DMA kernel
//     below);
//   - otherwise (ragged token counts in the weight-gradient GEMMs): MFMA
//     v_mfma_f32_32x32x16_bf16, K-tile 64, double-buffered LDS, loads staged
//     through registers with zero fill; an M- or N-contiguous operand is
//     loaded as 8x8 blocks and transposed in registers on its way into LDS.
// The MFMA is issued with the roles of the operands swapped (the N tile as
// MFMA "A"), so each lane ends up holding four consecutive output columns of
// one row.  The DMA kernel stages its accumulators through LDS before the
// epilogue so that the epilogue's loads and stores cover whole lines; the
// register-staged kernel applies the epilogue from the accumulator layout.
//
// The epilogues carry the block's elementwise work (MegaScale Section 3.3
// fuses these fine-grained ops): in-projection bias + GeLU writing both U and
// G, out-projection bias + residual, and the GeLU derivative in the backward
// pass.
//
// fp32 path: a plain LDS-tiled SIMT kernel with the same epilogues.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace pb {
namespace {

// ------------------------------------------------------------- epilogues
// Four consecutive output columns n..n+3 of row m.  GT: tanh form of GeLU.
template <typename T, Epi EPI, bool GT>
PB_DEV void epi_store4(const EpiArgs& ep, int m, int n, const float* v) {
  if constexpr (EPI == Epi::StoreF32) {
    store4((float*)ep.out + (size_t)m * ep.ld_out + n, v);
  } else if constexpr (EPI == Epi::LnGrad) {
    store4((T*)ep.out + (size_t)m * ep.ld_out + n, v);
  } else if constexpr (EPI == Epi::BiasGelu) {
    float b[4], z[4];
    load4((const T*)ep.bias + n, b);
#pragma unroll
    for (int e = 0; e < 4; ++e) z[e] = v[e] + b[e];
    store4((T*)ep.out + (size_t)m * ep.ld_out + n, z);
    if (n >= ep.split) {
      float g[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) g[e] = gelu<GT>(z[e]);
      store4((T*)ep.out2 + (size_t)m * ep.ld_out2 + (n - ep.split) + ep.col2, g);
    }
  } else if constexpr (EPI == Epi::BiasResid) {
    float b[4], r[4], o[4];
    load4((const T*)ep.bias + n, b);
    load4((const T*)ep.resid + (size_t)m * ep.ld_out + n, r);
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = v[e] + b[e] + r[e];
    store4((T*)ep.out + (size_t)m * ep.ld_out + n, o);
  } else {  // DgeluSplit
    if (n < ep.split) {
      store4((T*)ep.out + (size_t)m * ep.ld_out + n, v);
    } else {
      const size_t off = (size_t)m * ep.ld_out2 + (n - ep.split) + ep.col2;
      float u[4], o[4];
      load4((const T*)ep.aux + off, u);
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = v[e] * gelu_grad<GT>(u[e]);
      store4((T*)ep.out2 + off, o);
    }
  }
}

// LnGrad: the LayerNorm backward's row terms of four columns n..n+3 of row m,
// added to s1 (sum g) and s2 (sum g xhat), g = gamma dh.
template <typename T>
PB_DEV void ln_terms4(const EpiArgs& ep, int m, int n, const float* v, float mu, float rs,
                      float& s1, float& s2) {
  float gm[4], xv[4];
  load4((const T*)ep.bias + n, gm);
  load4((const T*)ep.aux + (size_t)m * ep.ld_out + n, xv);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float g = gm[e] * v[e];
    s1 += g;
    s2 += g * ((xv[e] - mu) * rs);
  }
}

// --------------------------------------------------------- bf16 MFMA GEMM
// 256 x 256 output tile, K-tile 64, eight waves in a 4 (m) x 2 (n) grid, each
// wave 64 x 128 (2 x 4 MFMA blocks of 32 x 32); two waves per SIMD hide each
// other's LDS and global latency.
constexpr int kBM = 256, kBN = 256, kBK = 64;
constexpr int kWavesM = 4, kWavesN = 2;
constexpr int kThreads = 64 * kWavesM * kWavesN;
constexpr int kWTM = kBM / kWavesM, kWTN = kBN / kWavesN;
constexpr int kTM = kWTM / 32, kTN = kWTN / 32;
constexpr int kTileBytes = kBM * kBK * 2;  // one operand tile (32 KB)
// CUs of MI355X; the DMA kernels' 128 KB of LDS allows one workgroup per CU.
constexpr int kCUs = 256;

// 16-byte chunk c (0..7) of LDS row `row` lives at physical chunk swz(row, c).
PB_DEV int swz(int row, int c) { return c ^ ((row ^ (row >> 3)) & 7); }

// Tile order.  Workgroup b runs on XCD b % 8; xcd_remap gives each XCD a
// contiguous run of logical ids, and tile_of walks logical ids in groups of G
// tile-rows, so concurrently running workgroups on one XCD share operand
// strips in its L2.  The LDS-DMA GEMMs take G = tile_group(epilogue): groups
// of 4 rows (a 32-workgroup XCD share spans 4 x 8 tiles) measured faster for
// the backward's GEMMs and the in-projection, groups of 8 for the
// out-projection (BiasResid); groups of 2 or 16 were slower for all.
PB_DEV int xcd_remap(int bid, int n) {
  const int q = n / 8, r = n % 8, x = bid % 8;
  return x * q + min(x, r) + bid / 8;
}
constexpr int tile_group(Epi e) { return e == Epi::BiasResid ? 8 : 4; }
template <int G = 8>
PB_DEV void tile_of(int lid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int per_group = G * tiles_n;
  const int group = lid / per_group;
  const int first_m = group * G;
  const int gsize = min(tiles_m - first_m, G);
  const int in_group = lid - group * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}
PB_DEV void tile_coords(int tiles_m, int tiles_n, int& tm, int& tn) {
  tile_of(xcd_remap(blockIdx.x, tiles_m * tiles_n), tiles_m, tiles_n, tm, tn);
}

// Epilogue of one wave's 64 x 128 block of a 256 x 256 tile.  acc[i][j][4 jj +
// e] is C(m, n) with m = mw + 32 i + (lane & 31), n = nw + 32 j + 8 jj +
// 4 (lane >> 5) + e.  For LnGrad, lanes l and l ^ 32 together hold all 128
// columns of a row, 64 per column group j / 2: their row terms are summed
// across the pair and written once per (row, group).
template <Epi EPI, bool GT>
PB_DEV void wave_epilogue(const EpiArgs& ep, const f32x16 (&acc)[kTM][kTN], int mw, int nw,
                          int M, int N, int fr, int fh) {
#pragma unroll
  for (int i = 0; i < kTM; ++i) {
    const int m = mw + 32 * i + fr;
    const bool mok = m < M;
    float s1[kTN / 2], s2[kTN / 2], mu = 0.f, rs = 0.f;
    if constexpr (EPI == Epi::LnGrad) {
#pragma unroll
      for (int h = 0; h < kTN / 2; ++h) s1[h] = s2[h] = 0.f;
      if (mok) {
        mu = ep.mean[m];
        rs = ep.rstd[m];
      }
    }
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int n = nw + 32 * j + 8 * jj + 4 * fh;
        if (mok && n < N) {
          float v[4] = {acc[i][j][4 * jj], acc[i][j][4 * jj + 1], acc[i][j][4 * jj + 2],
                        acc[i][j][4 * jj + 3]};
          epi_store4<bf16, EPI, GT>(ep, m, n, v);
          if constexpr (EPI == Epi::LnGrad) ln_terms4<bf16>(ep, m, n, v, mu, rs, s1[j / 2], s2[j / 2]);
        }
      }
    if constexpr (EPI == Epi::LnGrad) {
#pragma unroll
      for (int h = 0; h < kTN / 2; ++h) {
        s1[h] += __shfl_xor(s1[h], 32, 64);
        s2[h] += __shfl_xor(s2[h], 32, 64);
        const int n = nw + 64 * h;  // group start (a multiple of 64)
        if (fh == 0 && mok && n < N)
          ep.rowpart[(size_t)m * ep.rowpart_ld + n / 64] = make_float2(s1[h], s2[h]);
      }
    }
  }
}

// One 256 x 64 operand tile, global -> registers -> LDS.
// KC: K-contiguous operand, row r of the tile at X[(R0 + r) * ld + k]: each
//     thread moves four 16-byte chunks (rows past Rmax are clamped: their
//     results are never stored).
// else MN-contiguous, X[k * ld + R0 + r]: each thread moves a 4 (k) x 8 (mn)
//     piece and transposes it into eight 8-byte LDS writes.
// k past K reads as zero.  Loads are unconditional (address clamped, value
// selected) so the loop body stays branch-free.
template <bool KC>
struct TileLoader {
  u32x4 r[4];
  uint32_t ok;  // bit i: r[i] is in range (else it is stored as zero)

  // The zero-fill select is applied in store(), not here: consuming the
  // loaded registers right away would make the compiler wait for the loads
  // before the MFMAs of the current tile instead of overlapping them.
  PB_DEV void load(const bf16* __restrict__ X, int ld, int R0, int Rmax, int k0, int K) {
    const int tid = threadIdx.x;
    ok = 0;
    if constexpr (KC) {
      const int c = tid & 7;
      const int k = k0 + 8 * c;
      const bool kok = k < K;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int row = R0 + (tid >> 3) + 64 * i;
        row = row < Rmax ? row : Rmax - 1;
        r[i] = *reinterpret_cast<const u32x4*>(X + (size_t)row * ld + (kok ? k : 0));
        ok |= (uint32_t)kok << i;
      }
    } else {
      const int col = R0 + 8 * (tid & 31);
      const int kq = tid >> 5;  // 0..15
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int k = k0 + 4 * kq + j;
        const bool in = k < K && col < Rmax;
        r[j] = *reinterpret_cast<const u32x4*>(X + (in ? (size_t)k * ld + col : 0));
        ok |= (uint32_t)in << j;
      }
    }
  }

  PB_DEV void store(unsigned char* __restrict__ lds) const {
    const int tid = threadIdx.x;
    u32x4 v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = ((ok >> i) & 1) ? r[i] : u32x4{0, 0, 0, 0};
    if constexpr (KC) {
      const int c = tid & 7;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = (tid >> 3) + 64 * i;
        *reinterpret_cast<u32x4*>(lds + row * 128 + swz(row, c) * 16) = v[i];
      }
    } else {
      const int mb = tid & 31, kq = tid >> 5;
      const int c = kq >> 1, half = kq & 1;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int q = i >> 1;
        uint32_t w0, w1;
        if (i & 1) {
          w0 = (v[0][q] >> 16) | (v[1][q] & 0xffff0000u);
          w1 = (v[2][q] >> 16) | (v[3][q] & 0xffff0000u);
        } else {
          w0 = (v[0][q] & 0xffffu) | (v[1][q] << 16);
          w1 = (v[2][q] & 0xffffu) | (v[3][q] << 16);
        }
        const int row = 8 * mb + i;
        *reinterpret_cast<u32x2*>(lds + row * 128 + swz(row, c) * 16 + half * 8) = u32x2{w0, w1};
      }
    }
  }
};

template <bool AK, bool BK, Epi EPI, bool GT>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_kernel(const bf16* __restrict__ A,
                                                                int lda,
                                                                const bf16* __restrict__ B,
                                                                int ldb, int M, int N, int K,
                                                                EpiArgs ep) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  // stage s: A tile at smem + 2 s * kTileBytes, B tile right after it
  auto lds_a = [&](int s) { return smem + (2 * s) * kTileBytes; };
  auto lds_b = [&](int s) { return smem + (2 * s + 1) * kTileBytes; };

  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = (N + kBN - 1) / kBN;
  int tm, tn;
  tile_coords(tiles_m, tiles_n, tm, tn);
  const int m0 = tm * kBM, n0 = tn * kBN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = (wave % kWavesM) * kWTM, wn = (wave / kWavesM) * kWTN;

  f32x16 acc[kTM][kTN];
#pragma unroll
  for (int i = 0; i < kTM; ++i)
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  TileLoader<AK> la;
  TileLoader<BK> lb;
  const int nk = (K + kBK - 1) / kBK;
  la.load(A, lda, m0, M, 0, K);
  lb.load(B, ldb, n0, N, 0, K);
  la.store(lds_a(0));
  lb.store(lds_b(0));
  __syncthreads();

  const int fr = lane & 31, fh = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      la.load(A, lda, m0, M, (kt + 1) * kBK, K);
      lb.load(B, ldb, n0, N, (kt + 1) * kBK, K);
    }
    const u32x4* pa = reinterpret_cast<const u32x4*>(lds_a(cur));
    const u32x4* pb = reinterpret_cast<const u32x4*>(lds_b(cur));
    // fragments of k-step ks + 1 are read while the MFMAs of ks run
    bf16x8 fa[2][kTM], fb[2][kTN];
    auto read_frags = [&](int ks, int buf) {
      const int c = 2 * ks + fh;
#pragma unroll
      for (int i = 0; i < kTM; ++i) {
        const int row = wm + 32 * i + fr;
        fa[buf][i] = __builtin_bit_cast(bf16x8, pa[row * 8 + swz(row, c)]);
      }
#pragma unroll
      for (int j = 0; j < kTN; ++j) {
        const int row = wn + 32 * j + fr;
        fb[buf][j] = __builtin_bit_cast(bf16x8, pb[row * 8 + swz(row, c)]);
      }
    };
    read_frags(0, 0);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int b = ks & 1;
      if (ks + 1 < kBK / 16) read_frags(ks + 1, b ^ 1);
#pragma unroll
      for (int i = 0; i < kTM; ++i)
#pragma unroll
        for (int j = 0; j < kTN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[b][j], fa[b][i], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      la.store(lds_a(cur ^ 1));
      lb.store(lds_b(cur ^ 1));
    }
    __syncthreads();
  }

  wave_epilogue<EPI, GT>(ep, acc, m0 + wm, n0 + wn, M, N, fr, fh);
}

// ------------------------------------------- bf16 MFMA GEMM, LDS-DMA path
// Used when K is a multiple of 64.  The operand tiles go from global memory
// straight into LDS (global_load_lds_dwordx4: each lane's 16 bytes land at
// LDS base + 16 * lane), so there is no register staging and no LDS write
// instruction.  K-tiles of 64 (a K-contiguous row then spans whole 128-byte
// lines) through two LDS stages (2 x 64 KB).
//
// The main loop runs on v_mfma_f32_16x16x32_bf16: on random bf16 operands
// the chip holds ~2.0 GHz issuing it back to back, against ~1.65 GHz for
// v_mfma_f32_32x32x16_bf16 at the same FLOP rate per clock (a power limit,
// measured with MFMA-only loops), so the same schedule gets ~20% more clock.
// A wave's 64 x 128 block is 4 x 8 MFMA blocks of 16 x 16; a K-tile is two
// k-steps of 32, and each k-step's MFMAs are issued in two phases (N blocks
// 0-3, then 4-7).  Each wave keeps the fragments of both k-steps in registers
// and reads them two phases ahead, so a tile's last reads are issued before
// its second phase's MFMAs; the one workgroup barrier of the K-tile sits
// there.  After it the tile's stage is free for the loads of tile t + 2 and
// tile t + 1 is visible, whose first fragments are read while the second
// k-step multiplies: the matrix pipe keeps running through the barrier and
// the loads have a whole tile to land.
//
// A K-contiguous operand is stored K-major (128-byte rows, the 16-byte chunk
// index XOR-swizzled by the row); an MN-contiguous operand is stored MN-major,
// 64 k-rows of 512 bytes with the chunk index XOR-ed by 4 (k mod 4) and by
// 2 (k / 8 mod 2), and its MFMA fragments are read with ds_read_b64_tr_b16,
// which transposes 4 (k) x 16 (mn) blocks across a 16-lane group (the four
// groups of a wave read k-rows 8 apart).  Both patterns are free of bank
// conflicts (64 banks).  The DMA instructions are issued from inline assembly as scalar
// base + per-lane offset (no per-load address arithmetic) and waited for
// explicitly, so the compiler adds no conservative waits between them and the
// LDS reads of the other stage.
typedef short s16x4 __attribute__((ext_vector_type(4)));
#define PB_LDS __attribute__((address_space(3)))

constexpr int kDK = 64;                     // K-tile of the DMA path
constexpr int kStages = 2;
constexpr int kDTile = kBM * kDK * 2;       // one operand tile: 32 KB
constexpr int kPieces = kDTile / kThreads / 16;  // 1 KB DMA pieces per operand per wave: 4
static_assert(kBM == kBN && kPieces * 1024 * (kThreads / 64) == kDTile, "tile split over waves");
static_assert(kDK == kBK, "the DMA path's K-tile is the planning unit");

// Materialise a wave-uniform value in scalar registers at this point.
template <typename T>
PB_DEV void pin_sgpr(T v) {
  asm volatile("" ::"s"(v));
}

PB_DEV int swz_mn(int krow, int c) { return c ^ (4 * (krow & 3)) ^ (2 * ((krow >> 3) & 1)); }

template <int N>
PB_DEV void wait_dma() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }
// The wait for LDS (and scalar) loads is the compiler's own instruction
// (lgkmcnt(0), vmcnt and expcnt left open), so its wait bookkeeping knows
// that nothing counted by lgkmcnt is outstanding past the barrier; hidden
// inside the asm, a kernel-argument load issued earlier would look pending
// and force a full wait at the main loop's head.
PB_DEV void block_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);
  asm volatile("s_barrier" ::: "memory");
}

// Byte offset, from the operand tile's base (its first row, or first column,
// at the tile's k), of this lane's 16 bytes in DMA piece i of this wave.
// KC: row r of the tile at X[(R0 + r) * ld + k]; rows past Rmax are clamped
// (their results are never stored).  Else X[k * ld + R0 + c], columns past
// Rmax clamped the same way.
template <bool KC>
PB_DEV uint32_t dma_lane_off(int ld, int R0, int Rmax, int wave, int lane, int i) {
  const int p = wave * (kPieces * 1024) + i * 1024 + 16 * lane;
  if constexpr (KC) {
    const int row = p >> 7, c = swz(row, (p >> 4) & 7);
    const int r = min(R0 + row, Rmax - 1) - R0;
    return (uint32_t)(r * ld + 8 * c) * 2u;
  } else {
    const int krow = p >> 9, c = swz_mn(krow, (p >> 4) & 31);
    const int col = min(R0 + 8 * c, Rmax - 8) - R0;
    return (uint32_t)(krow * ld + col) * 2u;
  }
}

// MFMA fragment (8 bf16 along k) of tile row `row`, k-step ks, lane half h.
template <bool KC>
PB_DEV bf16x8 dma_frag(const unsigned char* lds_tile, int row, int ks, int h, int lane) {
  if constexpr (KC) {
    return *reinterpret_cast<const bf16x8*>(lds_tile + row * 128 + swz(row, 2 * ks + h) * 16);
  } else {
    // lane 4 j + q of a 16-lane group reads k-row kb + j, mn (row & ~15) + 4 q;
    // the transposing read hands lane i the four k values of mn (row & ~15) + i
    const int i = lane & 15;
    const int j = i >> 2, q = i & 3;
    const int mn = (row & ~15) + 4 * q;
    const int kb = 16 * ks + 8 * h;
    const int c = mn >> 3, off = (mn & 7) * 2;
    const int k1 = kb + j, k2 = kb + 4 + j;
    const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (PB_LDS s16x4*)(lds_tile + k1 * 512 + swz_mn(k1, c) * 16 + off));
    const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (PB_LDS s16x4*)(lds_tile + k2 * 512 + swz_mn(k2, c) * 16 + off));
    const bf16x4 a4 = __builtin_bit_cast(bf16x4, a), b4 = __builtin_bit_cast(bf16x4, b);
    return bf16x8{a4[0], a4[1], a4[2], a4[3], b4[0], b4[1], b4[2], b4[3]};
  }
}

// Fragment of v_mfma_f32_16x16x32_bf16 for the 16-row block at tile row
// `base` (a multiple of 16), k-step s (32 k) of the K-tile: lane l supplies
// row base + (l & 15) and its k values 32 s + 8 (l >> 4) .. + 7, i.e. the
// 16-byte chunk 4 s + (l >> 4) of that row.
template <bool KC>
PB_DEV bf16x8 dma_frag16(const unsigned char* lds_tile, int base, int s, int lane) {
  return dma_frag<KC>(lds_tile, base + (lane & 15), 2 * s + (lane >> 5), (lane >> 4) & 1, lane);
}

// A wave's 64 x 128 block as 16 x 16 MFMA blocks.  acc[i][j][e] is C(m, n)
// with m = mw + 16 i + (lane & 15), n = nw + 16 j + 4 (lane >> 4) + e (the N
// tile is the MFMA's "A" operand, so each lane holds four consecutive columns
// of one row).
constexpr int kTM16 = kWTM / 16, kTN16 = kWTN / 16;

// The epilogue of a wave's 64 x 128 block of the tile, staged through the
// wave's 16 KB of LDS so that every global access of the epilogue covers
// whole lines.  Per 32-row half, the lanes write their accumulators row-major
// (the 16-byte chunk index XOR-ed by the row), read them back as four
// consecutive columns of one row per lane (two rows per instruction), and
// apply the epilogue to those four columns: fp32 results go out as 512
// contiguous bytes of a row per 32 lanes, bf16 results and the bias,
// residual and GeLU inputs as 256.  Applied straight from the accumulator
// layout, each access would cover 8 to 32 bytes of 32 different rows.
// Weight gradients are written with non-temporal stores; K-slice partials
// (part_tile: ld kBN, no epilogue), which the reduction reads right after,
// with ordinary ones.  For LnGrad each 16-lane group holds one
// row's 64-column group and sums its row terms across the group.
// acc[i][j][4 jj + e] is row mw + 32 i + fr, column nw + 32 j + 8 jj + 4 fh +
// e.  All LDS reads of the main loop must be finished (block barrier) first.
constexpr int kEpiWaveLds = 32 * kWTN * 4;  // one half: 16 KB
static_assert(kEpiWaveLds * kWavesM * kWavesN <= 4 * kTileBytes, "epilogue staging fits");
template <Epi EPI, bool GT>
PB_DEV void wave_epilogue_lds(const EpiArgs& ep, float* __restrict__ part_tile,
                              const f32x4 (&acc)[kTM16][kTN16], int mw, int nw, int M, int N,
                              int lane, unsigned char* buf) {
  const int c = lane & 31, hi = lane >> 5;
  const int n = nw + 4 * c;  // this lane's four columns, the same in every row
  const int ncl = min(n, N - 4);
  // inputs that depend only on the column, loaded once
  float b4[4] = {0.f, 0.f, 0.f, 0.f};
  if constexpr (EPI == Epi::BiasGelu || EPI == Epi::BiasResid || EPI == Epi::LnGrad)
    if (!part_tile) load4<bf16>((const bf16*)ep.bias + ncl, b4);
  const bool dg_aux = EPI == Epi::DgeluSplit && ep.split < N;  // any GeLU' column at all
#pragma unroll
  for (int i = 0; i < kWTM / 32; ++i) {
    // rows 16 ii + (lane & 15) of the half, 16-byte column chunk 4 j + (lane >> 4)
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int j = 0; j < kTN16; ++j) {
        const int rr = 16 * ii + (lane & 15), cw = 4 * j + (lane >> 4);
        *reinterpret_cast<f32x4*>(buf + rr * (kWTN * 4) + ((cw ^ rr) & 31) * 16) = acc[2 * i + ii][j];
      }
    const int m0h = mw + 32 * i;  // first row of this half
    // Per-row inputs of the half, all issued before any result is stored (a
    // wait for a load also waits for every earlier store): the residual,
    // GeLU input or LayerNorm input of this lane's four columns in each of
    // its 16 rows, at clamped addresses; LayerNorm statistics one row per
    // lane, broadcast below.
    u32x2 in2[16];
    float mu_l = 0.f, rs_l = 0.f;
    if (!part_tile) {
      if constexpr (EPI == Epi::BiasResid || EPI == Epi::LnGrad) {
        const bf16* src = (const bf16*)(EPI == Epi::BiasResid ? ep.resid : ep.aux);
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          const int mc = min(m0h + 2 * t + hi, M - 1);
          in2[t] = *reinterpret_cast<const u32x2*>(src + (size_t)mc * ep.ld_out + ncl);
        }
      }
      if constexpr (EPI == Epi::DgeluSplit) {
        if (ep.delta && n < ep.split) {
          // the attention output O of this lane's four columns, for delta
#pragma unroll
          for (int t = 0; t < 16; ++t) {
            const int mc = min(m0h + 2 * t + hi, M - 1);
            in2[t] = *reinterpret_cast<const u32x2*>((const bf16*)ep.o_rows +
                                                     (size_t)mc * ep.ld_o_rows + ncl);
          }
        } else if (dg_aux) {
          const int col = max(ncl - ep.split, 0) + ep.col2;
#pragma unroll
          for (int t = 0; t < 16; ++t) {
            const int mc = min(m0h + 2 * t + hi, M - 1);
            in2[t] = *reinterpret_cast<const u32x2*>((const bf16*)ep.aux +
                                                     (size_t)mc * ep.ld_out2 + col);
          }
        }
      }
      if constexpr (EPI == Epi::LnGrad) {
        const int mr = min(m0h + c, M - 1);
        mu_l = ep.mean[mr];
        rs_l = ep.rstd[mr];
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int r = 2 * t + hi;
      const f32x4 v = *reinterpret_cast<const f32x4*>(buf + r * (kWTN * 4) + ((c ^ r) & 31) * 16);
      const int m = m0h + r;
      const bool ok = m < M && n < N;
      if (part_tile) {
        if (ok) *reinterpret_cast<f32x4*>(part_tile + m * kBN + n) = v;
        continue;
      }
      float o[4];
      if constexpr (EPI == Epi::StoreF32) {
        if (ok)
          __builtin_nontemporal_store(
              v, reinterpret_cast<f32x4*>((float*)ep.out + (size_t)m * ep.ld_out + n));
      } else if constexpr (EPI == Epi::BiasGelu) {
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = v[e] + b4[e];
        if (ok) {
          store4((bf16*)ep.out + (size_t)m * ep.ld_out + n, o);
          if (n >= ep.split) {
            float g[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) g[e] = gelu<GT>(o[e]);
            store4((bf16*)ep.out2 + (size_t)m * ep.ld_out2 + (n - ep.split) + ep.col2, g);
          }
        }
      } else if constexpr (EPI == Epi::BiasResid) {
        const float rr[4] = {lo_bf(in2[t][0]), hi_bf(in2[t][0]), lo_bf(in2[t][1]),
                             hi_bf(in2[t][1])};
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = v[e] + b4[e] + rr[e];
        if (ok) store4((bf16*)ep.out + (size_t)m * ep.ld_out + n, o);
      } else if constexpr (EPI == Epi::DgeluSplit) {
        if (n < ep.split) {
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = v[e];
          if (ok) store4((bf16*)ep.out + (size_t)m * ep.ld_out + n, o);
          if (ep.delta) {
            // rowsum of dO * O over each head's columns (dO as stored), the
            // head's lanes (hd / 4 of them) summed across
            const float ov[4] = {lo_bf(in2[t][0]), hi_bf(in2[t][0]), lo_bf(in2[t][1]),
                                 hi_bf(in2[t][1])};
            float sd = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) sd += bf2f(f2bf(v[e])) * ov[e];
            const int gl = ep.delta_hd >> 2;  // lanes per head: 32 or 16
            for (int off = 1; off < gl; off <<= 1) sd += __shfl_xor(sd, off, 64);
            if ((c & (gl - 1)) == 0 && ok) {
              const int b = m / ep.delta_seq, tt = m - b * ep.delta_seq;
              ep.delta[((size_t)b * ep.delta_heads + n / ep.delta_hd) * ep.delta_seq + tt] = sd;
            }
          }
        } else {
          const float u[4] = {lo_bf(in2[t][0]), hi_bf(in2[t][0]), lo_bf(in2[t][1]),
                              hi_bf(in2[t][1])};
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = v[e] * gelu_grad<GT>(u[e]);
          if (ok)
            store4((bf16*)ep.out2 + (size_t)m * ep.ld_out2 + (n - ep.split) + ep.col2, o);
        }
      } else {  // LnGrad: dh, and the row terms of this lane's 64-column group
        const float xv[4] = {lo_bf(in2[t][0]), hi_bf(in2[t][0]), lo_bf(in2[t][1]),
                             hi_bf(in2[t][1])};
        const float mu_a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mu_l), 2 * t));
        const float mu_b =
            __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mu_l), 2 * t + 1));
        const float rs_a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(rs_l), 2 * t));
        const float rs_b =
            __int_as_float(__builtin_amdgcn_readlane(__float_as_int(rs_l), 2 * t + 1));
        const float mu = hi ? mu_b : mu_a, rs = hi ? rs_b : rs_a;
        float s1 = 0.f, s2 = 0.f;
        if (ok) {
          const float dh[4] = {v[0], v[1], v[2], v[3]};
          store4((bf16*)ep.out + (size_t)m * ep.ld_out + n, dh);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float g = b4[e] * v[e];
            s1 += g;
            s2 += g * ((xv[e] - mu) * rs);
          }
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) {
          s1 += __shfl_xor(s1, off, 64);
          s2 += __shfl_xor(s2, off, 64);
        }
        if ((c & 15) == 0 && ok)  // n is the group's first column
          ep.rowpart[(size_t)m * ep.rowpart_ld + n / 64] = make_float2(s1, s2);
      }
    }
  }
}

// Work items: the first n_full workgroups compute whole tiles (logical ids
// 0 .. n_full - 1); the remaining tail * splits workgroups each compute one
// K-slice of one of the last `tail` tiles and store its fp32 partial tile
// (256 x 256, row-major) to part, for splitk_reduce.
// One work item of the DMA GEMM: K-tiles [kt0, kt1) of output tile lid
// (slice >= 0: one K-slice of tail tile lid, whose fp32 partial tile goes to
// part for splitk_reduce).
// Sum of a fragment's eight bf16 values, added to acc in fp32.
PB_DEV float sum_bf16x8(const bf16x8& p, float acc) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 8; i += 2)
    acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2_t{p[i], p[i + 1]}, one, acc, false);
  return acc;
}

// RS (StoreF32 only): also the row sums of A over this work item's K-tiles,
// rowsum[m] = sum_k A(m, k), from the A fragments the MFMAs consume (the
// caller sets RS for the tiles of the first tile column only).
// Persistent launches pass qctr: thread 0 then takes the next ticket of that
// queue (*qticket) right after the main loop, so the atomic's latency is
// spent under the epilogue; and tid_in, the thread index the caller keeps
// out of the compiler's sight (see gemm_bf16_dma_pair_persistent).
template <bool AK, bool BK, Epi EPI, bool GT, bool RS = false>
PB_DEV void dma_gemm_item(const bf16* __restrict__ A, int lda, const bf16* __restrict__ B, int ldb,
                          int M, int N, const EpiArgs& ep, int lid, int slice, int kt0, int kt1,
                          int n_full, int splits, float* __restrict__ part,
                          int* __restrict__ qctr = nullptr, int* qticket = nullptr,
                          int tid_in = -1) {
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(PB_LDS unsigned char*)smem;
  auto a_off = [&](int s) { return (2 * s) * kDTile; };
  auto b_off = [&](int s) { return (2 * s + 1) * kDTile; };

  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = (N + kBN - 1) / kBN;
  int tm, tn;
  tile_of<tile_group(EPI)>(lid, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * kBM, n0 = tn * kBN;
  const int tid = tid_in >= 0 ? tid_in : (int)threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int wm = (wave % kWavesM) * kWTM, wn = (wave / kWavesM) * kWTN;

  // K-tiles [kt0, kt1) of this work item
  const int nt = kt1 - kt0;
  // Who moves which part of a K-tile, and when.  All eight waves issuing
  // their loads together right after the barrier stalls them: the CU's load
  // path takes the 64 KB of a K-tile in roughly a thousand cycles, and a wave
  // whose load cannot be queued stops issuing, MFMAs included, while the
  // second wave of each SIMD, already behind the first, falls further behind
  // (per-phase clock stamps: ~1000 cycles between the two waves of a SIMD,
  // ~2800 cycles per K-tile against 2048 of matrix work).  Measured best:
  //  - both operands K-contiguous: every wave moves its own 4 KB of each
  //    operand, A of tile t + 2 right after the barrier of tile t and B of
  //    tile t + 1 at the start of tile t;
  //  - otherwise (transposing fragment reads): the first wave of each SIMD
  //    (waves 0-3) moves both 4 KB regions of its SIMD, on the same schedule,
  //    and the second wave none, which also slows the leading wave down to
  //    its partner's pace.
  constexpr int kReg = BK ? 1 : 2;  // 4 KB regions per operand per issuing wave
  constexpr int kDmaPerTile = 2 * kReg * kPieces;
  const bool dma_wave = BK || wave < 4;
  auto region = [&](int r) { return BK ? wave : (wave & 3) + 4 * r; };
  uint32_t aoff[kReg * kPieces], boff[kReg * kPieces];
#pragma unroll
  for (int r = 0; r < kReg; ++r)
#pragma unroll
    for (int i = 0; i < kPieces; ++i) {
      aoff[r * kPieces + i] = dma_lane_off<AK>(lda, m0, M, region(r), lane, i);
      boff[r * kPieces + i] = dma_lane_off<BK>(ldb, n0, N, region(r), lane, i);
    }
  const bf16* abase = (AK ? A + (size_t)m0 * lda : A + m0) + (size_t)kt0 * (AK ? kDK : (size_t)kDK * lda);
  const bf16* bbase = (BK ? B + (size_t)n0 * ldb : B + n0) + (size_t)kt0 * (BK ? kDK : (size_t)kDK * ldb);
  const size_t astep = AK ? kDK : (size_t)kDK * lda;  // elements per K-tile
  const size_t bstep = BK ? kDK : (size_t)kDK * ldb;
  // this wave's pieces of one operand of tile t (half 0: A, half 1: B)
  auto issue_half = [&](int t, int half) {
    if (!dma_wave) return;
    const int s = t % kStages;
    const bf16* src = half == 0 ? abase + (size_t)t * astep : bbase + (size_t)t * bstep;
    const uint32_t dst0 = lds0 + (half == 0 ? a_off(s) : b_off(s));
#pragma unroll
    for (int r = 0; r < kReg; ++r)
#pragma unroll
      for (int i = 0; i < kPieces; ++i)
        dma16s(src, half == 0 ? aoff[r * kPieces + i] : boff[r * kPieces + i],
               __builtin_amdgcn_readfirstlane(dst0 + region(r) * (kPieces * 1024) + i * 1024));
  };
  auto issue = [&](int t) {
    issue_half(t, 0);
    issue_half(t, 1);
  };

  f32x4 acc[kTM16][kTN16];
#pragma unroll
  for (int i = 0; i < kTM16; ++i)
#pragma unroll
    for (int j = 0; j < kTN16; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Phase p (0..7) of a K-tile: k-step s = p / 4 (32 k), N blocks 2 (p % 4)
  // and 2 (p % 4) + 1, eight MFMAs.  Fragments are read kLook phases before
  // the phase that first uses them: the A blocks of k-step s with the batch
  // of phase 4 s, each pair of N blocks with its own phase's batch.  The
  // reads of a K-tile's last phase are issued kLook phases before its end;
  // the one workgroup barrier of the K-tile follows them, after which the
  // tile's stage takes A of tile t + 2 (and, from the start of tile t + 1,
  // B) while the next tile's first fragments are read.  With kLook = 2 at
  // most 14 fragments are live (56 registers beside the 128 of the
  // accumulators) and a load has most of a K-tile to land.
  constexpr int kPh = 8, kLook = 2;
  static_assert(kLook >= 2 && kLook < kPh, "DMA halves are issued after the barrier");
  bf16x8 fa[2][kTM16], fb[2][kTN16];
  auto read_frags = [&](int t, int p) {
    const int st = t % kStages, ks = p >> 2, r = p & 3;
    const unsigned char* pa = smem + a_off(st);
    const unsigned char* pb = smem + b_off(st);
    if (r == 0) {
#pragma unroll
      for (int i = 0; i < kTM16; ++i) fa[ks][i] = dma_frag16<AK>(pa, wm + 16 * i, ks, lane);
    }
#pragma unroll
    for (int j = 2 * r; j < 2 * r + 2; ++j) fb[ks][j] = dma_frag16<BK>(pb, wn + 16 * j, ks, lane);
  };
  float rsum[kTM16];
#pragma unroll
  for (int i = 0; i < kTM16; ++i) rsum[i] = 0.f;
  auto mma = [&](auto P) {
    constexpr int p = decltype(P)::value, ks = p >> 2, j0 = 2 * (p & 3);
    if constexpr (RS && (p & 3) == 0) {
#pragma unroll
      for (int i = 0; i < kTM16; ++i) rsum[i] = sum_bf16x8(fa[ks][i], rsum[i]);
    }
#pragma unroll
    for (int i = 0; i < kTM16; ++i)
#pragma unroll
      for (int j = j0; j < j0 + 2; ++j)
        acc[i][j] =
            __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[ks][j], fa[ks][i], acc[i][j], 0, 0, 0);
    // alternate one MFMA and one LDS read (the batch of phase p + kLook; a
    // transposed fragment takes two reads) so the reads are in flight early
    // and the matrix pipe stays fed
    constexpr int pn = (p + kLook) % kPh;
    constexpr int kReads = ((pn & 3) == 0 ? (AK ? 1 : 2) * kTM16 : 0) + (BK ? 1 : 2) * 2;
    constexpr int kMfma = kTM16 * 2;
    constexpr int pairs = kReads < kMfma ? kReads : kMfma;
#pragma unroll
    for (int u = 0; u < pairs; ++u) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    if constexpr (kMfma > pairs) __builtin_amdgcn_sched_group_barrier(0x008, kMfma - pairs, 0);
    if constexpr (kReads > pairs) __builtin_amdgcn_sched_group_barrier(0x100, kReads - pairs, 0);
  };
  auto phase = [&](int t, auto P) {
    constexpr int p = decltype(P)::value;
    if constexpr (p == kPh - kLook) {
      // Every wave has issued (and with the barrier, finished) its reads of
      // tile t, so its stage can take tile t + 2; tile t + 1 has landed for
      // this wave, and after the barrier for all.
      wait_dma<0>();
      block_barrier();
      if (t + 2 < nt) issue_half(t + 2, 0);
    }
    // B of tile t + 1 (tiles 0 and 1 were issued whole before the loop)
    if constexpr (p == 0)
      if (t + 1 >= 2 && t + 1 < nt) issue_half(t + 1, 1);
    // the batch kLook phases ahead (past the last tile: a stale stage, unused)
    if constexpr (p + kLook < kPh) read_frags(t, p + kLook);
    else read_frags(t + 1, p + kLook - kPh);
    mma(P);
    // each phase its own scheduling region: otherwise the scheduler may move
    // a later phase's MFMA (whose fragments were just requested) to the
    // front and the wait for it stalls on every outstanding LDS read
    __builtin_amdgcn_sched_barrier(0);
  };

  // The epilogue's kernel arguments are fetched before the first barrier,
  // whose wait covers them: a scalar load still in flight at the main loop's
  // head would make the loop's first LDS wait a full one (scalar loads return
  // out of order), on every K-tile.
  pin_sgpr(ep.out), pin_sgpr(ep.ld_out), pin_sgpr(ep.out2), pin_sgpr(ep.ld_out2);
  pin_sgpr(ep.bias), pin_sgpr(ep.resid), pin_sgpr(ep.aux), pin_sgpr(ep.split);
  pin_sgpr(ep.col2), pin_sgpr(ep.mean), pin_sgpr(ep.rstd), pin_sgpr(ep.rowpart);
  pin_sgpr(ep.rowpart_ld), pin_sgpr(part), pin_sgpr(ep.o_rows), pin_sgpr(ep.ld_o_rows);
  pin_sgpr(ep.delta), pin_sgpr(ep.delta_seq), pin_sgpr(ep.delta_heads), pin_sgpr(ep.delta_hd);
  if (nt > 0) issue(0);
  if (nt > 1) issue(1);
  if (nt > 1) wait_dma<kDmaPerTile>();  // tile 0 landed; tile 1 may be in flight
  else wait_dma<0>();
  block_barrier();
  // batch by batch, as in the loop, so the wait at the loop's head (merged
  // over both ways in) can leave the later batches in flight
#pragma unroll
  for (int p = 0; p < kLook; ++p) {
    read_frags(0, p);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int t = 0; t < nt; ++t) {
    phase(t, std::integral_constant<int, 0>{});
    phase(t, std::integral_constant<int, 1>{});
    phase(t, std::integral_constant<int, 2>{});
    phase(t, std::integral_constant<int, 3>{});
    phase(t, std::integral_constant<int, 4>{});
    phase(t, std::integral_constant<int, 5>{});
    phase(t, std::integral_constant<int, 6>{});
    phase(t, std::integral_constant<int, 7>{});
  }

  block_barrier();  // every wave is done with the main loop's LDS
  if (qctr && tid == 0) *qticket = atomicAdd(qctr, 1);
  if constexpr (RS) {
    // lanes l, l + 16, l + 32, l + 48 hold the same row's k groups; the four
    // waves of the first tile column (wn = 0) cover the tile's 256 rows
#pragma unroll
    for (int i = 0; i < kTM16; ++i) {
      float v = rsum[i];
      v += __shfl_xor(v, 16, 64);
      v += __shfl_xor(v, 32, 64);
      const int m = m0 + wm + 16 * i + (lane & 15);
      if (wn == 0 && lane < 16 && m < M) ep.rowsum[m] = v;
    }
  }
  unsigned char* buf = smem + wave * kEpiWaveLds;
  if (slice >= 0) {
    // partial tile of one K-slice, stored whole (bounds are applied on reduce)
    float* pt = part + ((size_t)(lid - n_full) * splits + slice) * (kBM * kBN);
    wave_epilogue_lds<EPI, GT>(ep, pt, acc, wm, wn, kBM, kBN, lane, buf);
  } else {
    wave_epilogue_lds<EPI, GT>(ep, nullptr, acc, m0 + wm, n0 + wn, M, N, lane, buf);
  }
}

template <bool AK, bool BK, Epi EPI, bool GT>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_dma_kernel(const bf16* __restrict__ A,
                                                                    int lda,
                                                                    const bf16* __restrict__ B,
                                                                    int ldb, int M, int N, int K,
                                                                    EpiArgs ep, int n_full,
                                                                    int splits,
                                                                    float* __restrict__ part) {
  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = (N + kBN - 1) / kBN;
  const int nk_all = K / kBK;  // slices are planned in units of 64
  int lid, slice = -1, kt0 = 0, kt1 = nk_all;
  if ((int)blockIdx.x < n_full) {
    lid = xcd_remap(blockIdx.x, n_full);
  } else {
    const int tail = tiles_m * tiles_n - n_full;
    const int j = xcd_remap(blockIdx.x - n_full, tail * splits);
    lid = n_full + j / splits;
    slice = j % splits;
    const int chunk = (nk_all + splits - 1) / splits;
    kt0 = min(nk_all, slice * chunk);
    kt1 = min(nk_all, kt0 + chunk);
  }
  dma_gemm_item<AK, BK, EPI, GT>(A, lda, B, ldb, M, N, ep, lid, slice, kt0, kt1, n_full, splits,
                                 part);
}

// Two independent GEMMs in one launch, neither split: workgroups 0 ..
// tiles1 - 1 compute the first one's tiles, the rest the second one's.  With
// the longer-K GEMM first, the second one's short tiles fill the CUs the
// first leaves idle (a partial last round) and its own partial last round is
// shared with nothing else; run apart, each GEMM pays its own.
struct DmaGemm {
  const bf16* A;
  int lda;
  const bf16* B;
  int ldb;
  int M, N, K;
  EpiArgs ep;
};
template <bool AK1, bool BK1, Epi E1, bool AK2, bool BK2, Epi E2, bool GT>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_dma_pair(DmaGemm g1, int tiles1,
                                                                  DmaGemm g2, int tiles2) {
  const int b = (int)blockIdx.x;
  if (b < tiles1) {
    dma_gemm_item<AK1, BK1, E1, GT>(g1.A, g1.lda, g1.B, g1.ldb, g1.M, g1.N, g1.ep,
                                    xcd_remap(b, tiles1), -1, 0, g1.K / kBK, tiles1, 1, nullptr);
    return;
  }
  const int lid = xcd_remap(b - tiles1, tiles2);
  if constexpr (E2 == Epi::StoreF32) {
    // the second GEMM's row sums, when asked for, from its first tile column
    int tm, tn;
    tile_of<tile_group(E2)>(lid, (g2.M + kBM - 1) / kBM, (g2.N + kBN - 1) / kBN, tm, tn);
    if (g2.ep.rowsum && tn == 0) {
      dma_gemm_item<AK2, BK2, E2, GT, true>(g2.A, g2.lda, g2.B, g2.ldb, g2.M, g2.N, g2.ep, lid, -1,
                                            0, g2.K / kBK, tiles2, 1, nullptr);
      return;
    }
  }
  dma_gemm_item<AK2, BK2, E2, GT>(g2.A, g2.lda, g2.B, g2.ldb, g2.M, g2.N, g2.ep, lid, -1, 0,
                                  g2.K / kBK, tiles2, 1, nullptr);
}

// Persistent form of the pair launch: one workgroup per CU takes work items
// until none is left.  The items (the first GEMM's tiles, then the
// second's) are dealt to eight queues, one per XCD, each holding the tiles
// the launch above gives that XCD (xcd_remap); a workgroup reads its XCD
// from the hardware, takes items from that queue and, once it is empty,
// from the others.  So a slower XCD hands its last items to faster ones
// (workgroup clock stamps showed XCDs 5-9% apart in K-tile time, and the
// launch waiting on the slowest), and no workgroup pays a launch and
// prologue between items.  The queue heads are kQueueInts ints that must be
// zero when the launch starts (launch_queue_reset); the launch leaves them
// non-zero.  Results do not depend on which workgroup takes an item.
struct PairArgs {
  DmaGemm g1;
  int tiles1;
  DmaGemm g2;
  int tiles2;
  int* queue;
};
typedef const PairArgs __attribute__((address_space(4)))* PairArgsPtr;
// Items [queue_start, queue_start + queue_count) of n go to XCD q's queue.
PB_DEV int queue_start(int n, int q) { return q * (n / 8) + min(q, n % 8); }
PB_DEV int queue_count(int n, int q) { return n / 8 + (q < n % 8 ? 1 : 0); }
template <bool AK1, bool BK1, Epi E1, bool AK2, bool BK2, Epi E2, bool GT>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_dma_pair_persistent(PairArgs args) {
  __shared__ int s_item;
  const int tiles1 = args.tiles1, tiles2 = args.tiles2;
  int* const queue = args.queue;
  // XCC_ID hardware register (bits 3:0: the XCD this wave runs on)
  const int x = __builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 7;
  auto item_of = [&](int q, int i) {  // i-th item of queue q, or -1 past its end
    const int c1 = queue_count(tiles1, q);
    if (i < c1) return queue_start(tiles1, q) + i;
    if (i < c1 + queue_count(tiles2, q)) return tiles1 + queue_start(tiles2, q) + (i - c1);
    return -1;
  };
  // Wave 0: the item of a ticket of the own queue or, past its end, one taken
  // from the first other queue (in XCD order after x) whose head has not
  // passed its end; every failed take moves a head past its end, so the loop
  // ends.
  auto resolve = [&](int ticket) {
    const int lane = threadIdx.x & 63;
    int item = item_of(x, ticket);
    while (item < 0) {
      int left = 0;
      if (lane < 8)
        left = queue_count(tiles1, lane) + queue_count(tiles2, lane) -
               __hip_atomic_load(queue + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      unsigned long long m = __ballot(left > 0) & 0xffull;
      if (!m) break;
      m = ((m >> x) | (m << (8 - x))) & 0xffull;  // bit v: queue x + v
      const int q = (x + __builtin_ctzll(m)) & 7;
      int i = 0;
      if (lane == 0) i = atomicAdd(queue + q, 1);
      item = item_of(q, __shfl(i, 0, 64));
    }
    return item;
  };
  if (threadIdx.x < 64) {
    int t = 0;
    if (threadIdx.x == 0) t = atomicAdd(queue + x, 1);
    const int it = resolve(__shfl(t, 0, 64));
    if (threadIdx.x == 0) s_item = it;
  }
  __syncthreads();
  int item = __builtin_amdgcn_readfirstlane(s_item);
  while (item >= 0) {
    // Thread 0's s_item write for the next item comes after this item's
    // barriers, which every thread reaches only after reading s_item above.
    int ticket = 0;
    // The thread index and the GEMM descriptions are taken afresh for every
    // item (the descriptions by scalar loads of the kernel arguments), hidden
    // from the compiler by empty asm: otherwise it keeps what it derives from
    // them live across items, runs out of registers and spills, and a reload
    // before the main loop put a full memory wait into every K-tile.
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    // (PairArgs is the kernel's only argument, so it starts the segment)
    PairArgsPtr pa = (PairArgsPtr)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(pa));
    const PairArgs* ap = (const PairArgs*)pa;
    if (item < tiles1) {
      const DmaGemm g1 = ap->g1;
      dma_gemm_item<AK1, BK1, E1, GT>(g1.A, g1.lda, g1.B, g1.ldb, g1.M, g1.N, g1.ep, item, -1, 0,
                                      g1.K / kBK, tiles1, 1, nullptr, queue + x, &ticket, tid);
    } else {
      const DmaGemm g2 = ap->g2;
      const int lid = item - tiles1;
      bool done = false;
      if constexpr (E2 == Epi::StoreF32) {
        int tm, tn;
        tile_of<tile_group(E2)>(lid, (g2.M + kBM - 1) / kBM, (g2.N + kBN - 1) / kBN, tm, tn);
        if (g2.ep.rowsum && tn == 0) {
          dma_gemm_item<AK2, BK2, E2, GT, true>(g2.A, g2.lda, g2.B, g2.ldb, g2.M, g2.N, g2.ep,
                                                lid, -1, 0, g2.K / kBK, tiles2, 1, nullptr,
                                                queue + x, &ticket, tid);
          done = true;
        }
      }
      if (!done)
        dma_gemm_item<AK2, BK2, E2, GT>(g2.A, g2.lda, g2.B, g2.ldb, g2.M, g2.N, g2.ep, lid, -1, 0,
                                        g2.K / kBK, tiles2, 1, nullptr, queue + x, &ticket, tid);
    }
    if (threadIdx.x < 64) {
      const int it = resolve(__shfl(ticket, 0, 64));
      if (threadIdx.x == 0) s_item = it;
    }
    __syncthreads();
    item = __builtin_amdgcn_readfirstlane(s_item);
  }
}

__global__ void queue_reset_kernel(int* __restrict__ q, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) q[i] = 0;
}

// Sum of the K-slice partials of each tail tile, in slice order (so the
// result does not depend on timing), then the epilogue.  64 workgroups per
// tile, each thread four consecutive columns of one row.
template <Epi EPI, bool GT>
__global__ __launch_bounds__(256) void splitk_reduce(const float* __restrict__ part, int M, int N,
                                                     int n_full, int splits, EpiArgs ep) {
  const int tiles_m = (M + kBM - 1) / kBM, tiles_n = (N + kBN - 1) / kBN;
  const int t_local = blockIdx.x / 64;
  const int g = (blockIdx.x % 64) * 256 + threadIdx.x;  // 0 .. 16383
  const int row = g / (kBN / 4), col = (g % (kBN / 4)) * 4;
  int tm, tn;
  tile_of<tile_group(EPI)>(n_full + t_local, tiles_m, tiles_n, tm, tn);
  const int m = tm * kBM + row, n = tn * kBN + col;
  const bool ok = m < M && n < N;
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (ok) {
    const float* p = part + (size_t)t_local * splits * (kBM * kBN) + row * kBN + col;
    f32x4 sum = *reinterpret_cast<const f32x4*>(p);
    for (int sl = 1; sl < splits; ++sl)
      sum += *reinterpret_cast<const f32x4*>(p + (size_t)sl * kBM * kBN);
    v[0] = sum[0], v[1] = sum[1], v[2] = sum[2], v[3] = sum[3];
    epi_store4<bf16, EPI, GT>(ep, m, n, v);
  }
  if constexpr (EPI == Epi::LnGrad) {
    // a wave is one row of the tile; 16 lanes cover one 64-column group
    float s1 = 0.f, s2 = 0.f;
    if (ok) ln_terms4<bf16>(ep, m, n, v, ep.mean[m], ep.rstd[m], s1, s2);
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) {
      s1 += __shfl_xor(s1, off, 16);
      s2 += __shfl_xor(s2, off, 16);
    }
    if ((threadIdx.x & 15) == 0 && ok)
      ep.rowpart[(size_t)m * ep.rowpart_ld + n / 64] = make_float2(s1, s2);
  }
}

// ----------------------------------------------------------- fp32 SIMT GEMM
constexpr int kSB = 64, kSK = 16;

template <bool AK, bool BK, Epi EPI, bool GT>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int lda,
                                                       const float* __restrict__ B, int ldb,
                                                       int M, int N, int K, EpiArgs ep) {
  __shared__ float as[kSK][kSB + 4];
  __shared__ float bs[kSK][kSB + 4];
  const int m0 = blockIdx.y * kSB, n0 = blockIdx.x * kSB;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += kSK) {
    for (int e = threadIdx.x; e < kSB * kSK; e += 256) {
      const int r = e / kSK, kk = e % kSK;  // r: m or n within the tile
      const int k = k0 + kk;
      const int m = m0 + r, n = n0 + r;
      float av = 0.f, bv = 0.f;
      if (k < K && m < M) av = AK ? A[(size_t)m * lda + k] : A[(size_t)k * lda + m];
      if (k < K && n < N) bv = BK ? B[(size_t)n * ldb + k] : B[(size_t)k * ldb + n];
      as[kk][r] = av;
      bs[kk][r] = bv;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kSK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = as[kk][ty * 4 + i];
        b[i] = bs[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i, n = n0 + tx * 4;
    const bool ok = m < M && n < N;
    if (ok) epi_store4<float, EPI, GT>(ep, m, n, acc[i]);
    if constexpr (EPI == Epi::LnGrad) {
      // the 16 lanes tx = 0..15 of a row cover its 64-column group n0 .. n0 + 63
      float s1 = 0.f, s2 = 0.f;
      if (ok) ln_terms4<float>(ep, m, n, acc[i], ep.mean[m], ep.rstd[m], s1, s2);
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) {
        s1 += __shfl_xor(s1, off, 16);
        s2 += __shfl_xor(s2, off, 16);
      }
      if (tx == 0 && m < M && n0 < N)
        ep.rowpart[(size_t)m * ep.rowpart_ld + n0 / 64] = make_float2(s1, s2);
    }
  }
}

// The DMA path addresses a tile as scalar base + 32-bit lane offset.
bool dma_offsets_fit(bool ak, int lda, bool bk, int ldb) {
  auto fits = [](bool kc, int ld) {
    return (kc ? (long long)kBM : (long long)kDK) * ld * 2 < (1LL << 31);
  };
  return fits(ak, lda) && fits(bk, ldb);
}

template <bool AK, bool BK, Epi EPI, bool GT>
void gemm_dispatch_layout(Dt dt, const void* A, int lda, const void* B, int ldb, int M, int N,
                          int K, const EpiArgs& ep, float* split_ws, size_t split_ws_floats,
                          hipStream_t s) {
  if (dt == Dt::BF16) {
    const int tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
    const size_t lds = 4 * (size_t)kTileBytes;  // both kernels: 128 KB
    static_assert(kStages * 2 * kDTile == 4 * kTileBytes, "DMA path LDS");
    if (K % kBK == 0 && dma_offsets_fit(AK, lda, BK, ldb)) {
      SplitPlan sp = gemm_split_plan(dt, M, N, K);
      if (sp.tail > 0 && (!split_ws || split_ws_floats < gemm_split_floats(sp)))
        sp = SplitPlan{tiles, 0, 1};
      gemm_bf16_dma_kernel<AK, BK, EPI, GT><<<sp.n_full + sp.tail * sp.splits, kThreads, lds, s>>>(
          (const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, ep, sp.n_full, sp.splits, split_ws);
      if (sp.tail > 0)
        splitk_reduce<EPI, GT><<<sp.tail * 64, 256, 0, s>>>(split_ws, M, N, sp.n_full, sp.splits, ep);
    } else
      gemm_bf16_kernel<AK, BK, EPI, GT><<<tiles, kThreads, lds, s>>>(
          (const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, ep);
  } else {
    dim3 grid((N + kSB - 1) / kSB, (M + kSB - 1) / kSB);
    gemm_f32_kernel<AK, BK, EPI, GT><<<grid, 256, 0, s>>>((const float*)A, lda, (const float*)B,
                                                          ldb, M, N, K, ep);
  }
}

template <Epi EPI, bool GT>
void gemm_dispatch(Dt dt, bool ak, bool bk, const void* A, int lda, const void* B, int ldb,
                   int M, int N, int K, const EpiArgs& ep, float* ws, size_t wsf, hipStream_t s) {
  if (ak && bk) gemm_dispatch_layout<true, true, EPI, GT>(dt, A, lda, B, ldb, M, N, K, ep, ws, wsf, s);
  else if (ak) gemm_dispatch_layout<true, false, EPI, GT>(dt, A, lda, B, ldb, M, N, K, ep, ws, wsf, s);
  else if (bk) gemm_dispatch_layout<false, true, EPI, GT>(dt, A, lda, B, ldb, M, N, K, ep, ws, wsf, s);
  else gemm_dispatch_layout<false, false, EPI, GT>(dt, A, lda, B, ldb, M, N, K, ep, ws, wsf, s);
}

}  // namespace

SplitPlan gemm_split_plan(Dt dt, int M, int N, int K) {
  const int tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
  SplitPlan none{tiles, 0, 1};
  if (dt != Dt::BF16 || K % kBK != 0) return none;
  const int nk = K / kBK;
  const int n_full = tiles / kCUs * kCUs;
  const int tail = tiles - n_full;
  if (tail == 0) return none;
  if (n_full > 0) {
    // the last, partial wave: split its tiles so that it fills the chip once
    const int splits = std::min(kCUs / tail, nk);
    if (splits < 2) return none;
    return SplitPlan{n_full, tail, splits};
  }
  // Fewer tiles than CUs: split every tile along K when that is estimated
  // to be faster.  Cost in K-tile steps of one workgroup: waves x K-tiles per
  // slice, plus the reduction (a fixed launch cost and the fp32 partial
  // tiles written and read back, about 1/16 of a step each).
  auto cost = [&](int s) {
    const int waves = (tiles * s + kCUs - 1) / kCUs;
    const double c = (double)waves * ((nk + s - 1) / s);
    return s == 1 ? c : c + 3.0 + tiles * s / 16.0;
  };
  int best = 1;
  for (int s = 2; s <= std::min(16, nk); ++s)
    if (cost(s) < cost(best)) best = s;
  if (best < 2) return none;
  return SplitPlan{0, tiles, best};
}

size_t gemm_split_floats(const SplitPlan& p) {
  return (size_t)p.tail * p.splits * kBM * kBN;
}

GemmLaunch gemm_launch_of(Dt dt, int M, int N, int K) {
  GemmLaunch g;
  if (dt == Dt::BF16) {
    g.tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
    g.plan = gemm_split_plan(dt, M, N, K);
    g.workgroups = g.plan.n_full + g.plan.tail * g.plan.splits;
    g.threads = kThreads;
  } else {
    g.tiles = ((M + kSB - 1) / kSB) * ((N + kSB - 1) / kSB);
    g.plan = SplitPlan{g.tiles, 0, 1};
    g.workgroups = g.tiles;
    g.threads = 256;
  }
  return g;
}

bool gemm_pair_supported(Dt dt, const GemmSpec& g1, const GemmSpec& g2) {
  if (dt != Dt::BF16) return false;
  for (const GemmSpec* g : {&g1, &g2})
    if (g->M <= 0 || g->N <= 0 || g->K <= 0 || g->K % kBK ||
        !dma_offsets_fit(g->a_kcontig, g->lda, g->b_kcontig, g->ldb))
      return false;
  // the pairs of the block's backward pass: dC or dh (A K-contiguous, B
  // MN-contiguous) first, a weight gradient (both MN-contiguous, fp32) second
  return g1.a_kcontig && !g1.b_kcontig && (g1.epi == Epi::DgeluSplit || g1.epi == Epi::LnGrad) &&
         !g2.a_kcontig && !g2.b_kcontig && g2.epi == Epi::StoreF32;
}

void launch_queue_reset(int* queue, int n, hipStream_t s) {
  if (n > 0) queue_reset_kernel<<<1, 64, 0, s>>>(queue, n);
}

bool launch_gemm_pair(Dt dt, const GemmSpec& g1, const GemmSpec& g2, int* queue, hipStream_t s) {
  if (!gemm_pair_supported(dt, g1, g2)) return false;
  auto desc = [](const GemmSpec& g) {
    return DmaGemm{(const bf16*)g.A, g.lda, (const bf16*)g.B, g.ldb, g.M, g.N, g.K, g.ep};
  };
  auto tiles = [](const GemmSpec& g) {
    return ((g.M + kBM - 1) / kBM) * ((g.N + kBN - 1) / kBN);
  };
  const DmaGemm d1 = desc(g1), d2 = desc(g2);
  const int t1 = tiles(g1), t2 = tiles(g2);
  const size_t lds = 4 * (size_t)kTileBytes;
  // (the erf GeLU' form keeps the plain launch: its persistent build spills)
  if (queue && (g1.epi == Epi::LnGrad || g1.ep.gelu_tanh)) {
    const PairArgs pa{d1, t1, d2, t2, queue};
    const int grid = std::min(kCUs, t1 + t2);
    if (g1.epi == Epi::LnGrad)
      gemm_bf16_dma_pair_persistent<true, false, Epi::LnGrad, false, false, Epi::StoreF32, true>
          <<<grid, kThreads, lds, s>>>(pa);
    else
      gemm_bf16_dma_pair_persistent<true, false, Epi::DgeluSplit, false, false, Epi::StoreF32,
                                    true><<<grid, kThreads, lds, s>>>(pa);
    return true;
  }
  if (g1.epi == Epi::LnGrad)
    gemm_bf16_dma_pair<true, false, Epi::LnGrad, false, false, Epi::StoreF32, true>
        <<<t1 + t2, kThreads, lds, s>>>(d1, t1, d2, t2);
  else if (g1.ep.gelu_tanh)
    gemm_bf16_dma_pair<true, false, Epi::DgeluSplit, false, false, Epi::StoreF32, true>
        <<<t1 + t2, kThreads, lds, s>>>(d1, t1, d2, t2);
  else
    gemm_bf16_dma_pair<true, false, Epi::DgeluSplit, false, false, Epi::StoreF32, false>
        <<<t1 + t2, kThreads, lds, s>>>(d1, t1, d2, t2);
  return true;
}

void launch_gemm(Dt dt, Epi epi, bool a_kcontig, bool b_kcontig, const void* A, int lda,
                 const void* B, int ldb, int M, int N, int K, const EpiArgs& ep, float* split_ws,
                 size_t split_ws_floats, hipStream_t s) {
  const bool gt = ep.gelu_tanh != 0;
  float* w = split_ws;
  const size_t wf = split_ws_floats;
  switch (epi) {
    case Epi::StoreF32:
      gemm_dispatch<Epi::StoreF32, true>(dt, a_kcontig, b_kcontig, A, lda, B, ldb, M, N, K, ep, w, wf, s);
      break;
    case Epi::BiasGelu:
      if (gt) gemm_dispatch<Epi::BiasGelu, true>(dt, a_kcontig, b_kcontig, A, lda, B, ldb, M, N, K, ep, w, wf, s);
      else gemm_dispatch<Epi::BiasGelu, false>(dt, a_kcontig, b_kcontig, A, lda, B, ldb, M, N, K, ep, w, wf, s);
      break;
    case Epi::BiasResid:
      gemm_dispatch<Epi::BiasResid, true>(dt, a_kcontig, b_kcontig, A, lda, B, ldb, M, N, K, ep, w, wf, s);
      break;
    case Epi::DgeluSplit:
      if (gt) gemm_dispatch<Epi::DgeluSplit, true>(dt, a_kcontig, b_kcontig, A, lda, B, ldb, M, N, K, ep, w, wf, s);
      else gemm_dispatch<Epi::DgeluSplit, false>(dt, a_kcontig, b_kcontig, A, lda, B, ldb, M, N, K, ep, w, wf, s);
      break;
    case Epi::LnGrad:
      gemm_dispatch<Epi::LnGrad, true>(dt, a_kcontig, b_kcontig, A, lda, B, ldb, M, N, K, ep, w, wf, s);
      break;
  }
}

}  // namespace pb
