// MFMA tile engine for the LM-head contractions on gfx950.
//
//   C[m][n] = sum_k A[m][k] * B[n][k]      (fp32 accumulation)
//
// A workgroup of 256 threads (4 waves as 2 x 2) owns a 256 x 256 tile of C;
// each wave owns 128 x 128 as 4 x 4 MFMA 32x32 blocks held in 256 accumulator
// registers per lane. K advances in slabs of 128 bytes per row (64 bf16 or 32
// fp32 elements) through an LDS ring of kStages x (32 KB of A + 32 KB of B).
// Slabs are copied global -> LDS directly (global_load_lds_dwordx4: no staging
// registers, no LDS store instructions) kAhead slabs ahead of the MFMAs.
//
// Both operands are stored K-contiguous ([mn][k], row stride ld). LDS holds
// [mn][k] rows of eight 16-byte chunks with chunk c of row r at position
// c ^ ((r >> 1) & 7), so that the 16-byte fragment reads of sixteen
// consecutive lanes touch all 64 banks. The next slab is loaded into registers while the current
// one feeds the MFMAs, and fragments of K step s+1 are read from LDS while
// step s multiplies.
//
// Accumulator layout of v_mfma_f32_32x32x{16_bf16,2_f32} (block of 32 x 32):
// lane l, register r holds row (r & 3) + 8 * (r >> 2) + 4 * (l >> 5), column l & 31.
// Both operands feed chunk (2s + (l >> 5)) of the slab at step s, so each lane
// contributes the same k indices to A and B and the product is exact for any
// hardware ordering of k inside the instruction.
//
// Tile raster: one tile per workgroup. Blocks are dispatched round-robin over
// the 8 XCDs (block b runs on XCD b % 8). Every 256 consecutive blocks form one
// "wave"; the 32 blocks of one XCD take SN N-tiles x (32 / SN) M-tiles, so
// blocks sharing an XCD's L2 share operand panels. In N-split mode the XCDs of
// a wave take different N-tiles of the same M-tiles (the wave covers 8 SN x
// 32/SN tiles); in M-split mode they take different M-tiles of the same N-tiles
// (SN x 256/SN), so an M-tile's rows are fetched by one XCD only.
#pragma once

#include "common.hpp"

namespace sao {

constexpr int kBM = 256;                        // rows of A per tile
constexpr int kBN = 256;                        // rows of B per tile
constexpr int kMI = 4;                          // 32-row MFMA blocks per wave along M
constexpr int kNI = 4;                          // 32-column MFMA blocks per wave along N
constexpr int kThreads = 256;                   // 4 waves: 2 along M x 2 along N
constexpr int kWavesN = 2;
constexpr int kRowChunks = 8;                   // 16-byte chunks per LDS row (128 bytes of K)
constexpr int kAChunks = kBM * kRowChunks;      // 32 KB
constexpr int kBChunks = kBN * kRowChunks;      // 32 KB
constexpr int kStages = 2;                      // LDS ring depth
constexpr int kAhead = kStages - 1;             // slabs copied ahead of the MFMAs
constexpr int kStageChunks = kAChunks + kBChunks;

struct GemmShape {
  const void* a;
  int64_t lda;
  int64_t m;               // valid rows of A (host bound)
  const void* b;
  int64_t ldb;
  int64_t n;               // valid rows of B (host bound)
  int64_t k;               // contraction length (host value)
  const int32_t* m_dev;    // optional device count overriding m
  const int32_t* n_dev;    // optional device count overriding n
  const int32_t* k_dev;    // optional device count overriding k
  int m_tiles;             // ceil(m / kBM) with the host bound
  int n_tiles;             // ceil(n / kBN) with the host bound
  int sn;                  // N tiles per XCD per raster wave (1, 2, 4 or 8)
  int msplit;              // 0: XCDs split the wave's N tiles; 1: XCDs split its M tiles
};

// Tiles of one raster wave (256 blocks) along N and along M.
__host__ __device__ inline int wave_n(const GemmShape& s) { return s.msplit ? s.sn : 8 * s.sn; }
__host__ __device__ inline int wave_m(const GemmShape& s) { return s.msplit ? 256 / s.sn : 32 / s.sn; }

// Number of 256-block raster waves times 256.
inline int gemm_grid(const GemmShape& s) {
  const int nw = (s.n_tiles + wave_n(s) - 1) / wave_n(s);
  const int mw = (s.m_tiles + wave_m(s) - 1) / wave_m(s);
  return nw * mw * 256;
}

// N-split: SN so that 8 SN N-tiles fill the N range with little waste.
inline int pick_sn(int n_tiles) {
  if (n_tiles % 32 == 0 || n_tiles > 96) return 4;
  if (n_tiles % 16 == 0) return 2;
  return 1;
}

// M-split: all of a narrow N range per XCD (up to 8 tiles).
inline int pick_sn_msplit(int n_tiles) {
  return n_tiles >= 8 ? 8 : (n_tiles >= 4 ? 4 : (n_tiles >= 2 ? 2 : 1));
}

template <class E>
struct Mma;

template <>
struct Mma<BF16> {
  __device__ __forceinline__ static void run(f32x16_t& acc, const v4u& a, const v4u& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};

template <>
struct Mma<F32> {
  __device__ __forceinline__ static void run(f32x16_t& acc, const v4u& a, const v4u& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  }
};

__device__ __forceinline__ v4u zero4() { return v4u{0u, 0u, 0u, 0u}; }

// LDS position of 16-byte chunk c of tile row r. The LDS serves 16 lanes of a
// 16-byte access per cycle across 64 banks (256 bytes, two 128-byte rows), so
// the 16 rows read by lanes 0-15 (and the 2 rows written by them) must land on
// 16 distinct (row parity, chunk) pairs: XOR with (r >> 1) & 7 does that.
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r >> 1) & 7); }

// Direct copy of 16 bytes per lane from global memory (uniform base `g` plus the
// lane's byte offset `off`) into LDS: lane l writes LDS bytes [m0 + 16 l, +16),
// m0 being the wave-uniform LDS byte address `lds_addr`. Issued as inline
// assembly so that the compiler does not insert its conservative full waits
// before every LDS read; completion is tracked with explicit vmcnt waits.
__device__ __forceinline__ void dma16(const void* g, uint32_t off, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(g), "s"(lds_addr)
               : "memory", "m0");
}

// This wave's copies except the N most recent have landed in LDS, its LDS
// reads have returned, then the workgroup barrier: afterwards every wave's
// copies of the next slab are visible and the stage read before is free.
template <int N>
__device__ __forceinline__ void wait_copies_barrier() {
  if constexpr (N == 0)
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  else
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(N) : "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Fragments of one K16 step (bf16; K8 for fp32): kMI rows of A, kNI rows of B.
struct Frags {
  v4u a[kMI];
  v4u b[kNI];
};

// Rows read by a lane differ by multiples of 32, which leaves (row >> 1) & 7 and
// hence the swizzle unchanged: one LDS address per operand and K step, the
// blocks at immediate offsets.
__device__ __forceinline__ void read_frags(Frags& f, const v4u* la, const v4u* lb, int s, int wm, int wn,
                                           int lane, int c_valid) {
  const int r32 = lane & 31;
  const int c = 2 * s + (lane >> 5);
  const int pc = c ^ ((r32 >> 1) & 7);
  const v4u* pa = la + (wm * (kBM / 2) + r32) * kRowChunks + pc;
  const v4u* pb = lb + (wn * (kBN / kWavesN) + r32) * kRowChunks + pc;
#pragma unroll
  for (int i = 0; i < kMI; ++i) f.a[i] = pa[i * 32 * kRowChunks];
#pragma unroll
  for (int j = 0; j < kNI; ++j) f.b[j] = pb[j * 32 * kRowChunks];
  if (c >= c_valid) {  // K tail of the last slab: chunk beyond K contributes nothing
#pragma unroll
    for (int i = 0; i < kMI; ++i) f.a[i] = zero4();
#pragma unroll
    for (int j = 0; j < kNI; ++j) f.b[j] = zero4();
  }
}

template <class E>
__device__ __forceinline__ void mma_step(f32x16_t (&acc)[kMI][kNI], const Frags& f) {
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < kNI; ++j) Mma<E>::run(acc[i][j], f.a[i], f.b[j]);
}

// LDS writes of this thread are complete, then the workgroup barrier. Unlike
// __syncthreads() this does not wait for outstanding global loads, which keeps
// the next slab's prefetch in flight across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Row index inside the 256-row tile of accumulator (mi, register r) for this lane.
__device__ __forceinline__ int acc_row(int wm, int mi, int r, int lane) {
  return wm * (kBM / 2) + mi * 32 + (r & 3) + 8 * (r >> 2) + 4 * (lane >> 5);
}
__device__ __forceinline__ int acc_col(int wn, int ni, int lane) {
  return wn * (kBN / kWavesN) + ni * 32 + (lane & 31);
}

// The generic kernel body: one 256 x 256 tile per workgroup. Epi provides:
//   begin(n0, wm, wn, lane)                 before the K loop
//   tile(acc, m0, n0, wm, wn, lane, lds)    after it (LDS is free)
//   finish(mt, n0, wm, wn, lane, lds)  last (LDS is free)
// Both operands are K-contiguous.
template <class E, class Epi>
__device__ __forceinline__ void gemm_body(const GemmShape& s, Epi& epi, v4u (*lds)[kStageChunks]) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / kWavesN;
  const int wn = wave % kWavesN;

  // Raster: block -> (N tile, M tile).
  const int b = blockIdx.x;
  const int sn = s.sn;
  const int nw = (s.n_tiles + wave_n(s) - 1) / wave_n(s);
  const int w = b >> 8;
  const int xcd = b & 7;
  const int slot = (b >> 3) & 31;
  int n_tile, mt;
  if (s.msplit) {
    n_tile = (w % nw) * sn + slot % sn;
    mt = (w / nw) * (256 / sn) + xcd * (32 / sn) + slot / sn;
  } else {
    n_tile = (w % nw) * 8 * sn + xcd * sn + slot % sn;
    mt = (w / nw) * (32 / sn) + slot / sn;
  }

  const int64_t n_valid = s.n_dev ? static_cast<int64_t>(*s.n_dev) : s.n;
  const int64_t m_valid = s.m_dev ? static_cast<int64_t>(*s.m_dev) : s.m;
  const int64_t k_valid = s.k_dev ? static_cast<int64_t>(*s.k_dev) : s.k;
  if (n_tile >= s.n_tiles || mt >= s.m_tiles) return;
  const int64_t n0 = static_cast<int64_t>(n_tile) * kBN;
  const int64_t m0 = static_cast<int64_t>(mt) * kBM;
  if (n0 >= n_valid || m0 >= m_valid || k_valid <= 0) return;

  constexpr int P = E::kPerChunk;
  const int64_t k_chunks = (k_valid + P - 1) / P;          // valid 16-byte chunks per row
  const int nk = static_cast<int>((k_chunks + 7) / 8);     // slabs of 8 chunks
  const int c_last = static_cast<int>(k_chunks - static_cast<int64_t>(nk - 1) * 8);  // 1..8

  epi.begin(n0, wm, wn, lane);

  f32x16_t acc[kMI][kNI];
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < kNI; ++j) acc[i][j] = f32x16_t{};

  const int esz = static_cast<int>(sizeof(typename E::storage));
  const char* a_base = static_cast<const char*>(s.a);
  const char* b_base = static_cast<const char*>(s.b);
  // Copy instruction q of this wave covers tile rows (wave * Q + q) * 8 + lane / 8;
  // lane l lands on physical chunk l & 7 of its row, so it fetches the logical
  // chunk that the swizzle maps there. Row offsets are 32-bit: operands are
  // limited to 2^31 elements on the host.
  constexpr int QA = kBM * kRowChunks / 64 / 4;  // copies per wave per A slab
  constexpr int QB = kBN * kRowChunks / 64 / 4;  // copies per wave per B slab
  uint32_t offa[QA], offb[QB];
  int lca[QA], lcb[QB];
#pragma unroll
  for (int q = 0; q < QA; ++q) {
    const int r = (wave * QA + q) * 8 + (lane >> 3);
    lca[q] = swz(r, lane & 7);
    int64_t row = m0 + r;
    row = row < m_valid ? row : m_valid - 1;
    offa[q] = static_cast<uint32_t>(row * s.lda * esz);
  }
#pragma unroll
  for (int q = 0; q < QB; ++q) {
    const int r = (wave * QB + q) * 8 + (lane >> 3);
    lcb[q] = swz(r, lane & 7);
    int64_t row = n0 + r;
    row = row < n_valid ? row : n_valid - 1;
    offb[q] = static_cast<uint32_t>(row * s.ldb * esz);
  }
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&lds[0][0]));
  // Issue the copies of slab kt into `stage` (chunks past K are clamped to the
  // last valid chunk; their fragments are zeroed in read_frags).
  auto copy_slab = [&](int kt, int stage) {
    const uint32_t sbase = lds0 + static_cast<uint32_t>(stage) * kStageChunks * 16;
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      int64_t c = static_cast<int64_t>(kt) * 8 + lca[q];
      c = c < k_chunks ? c : k_chunks - 1;
      dma16(a_base, offa[q] + static_cast<uint32_t>(c * P * esz),
            __builtin_amdgcn_readfirstlane(sbase + (wave * QA + q) * 1024));
    }
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      int64_t c = static_cast<int64_t>(kt) * 8 + lcb[q];
      c = c < k_chunks ? c : k_chunks - 1;
      dma16(b_base, offb[q] + static_cast<uint32_t>(c * P * esz),
            __builtin_amdgcn_readfirstlane(sbase + kAChunks * 16 + (wave * QB + q) * 1024));
    }
  };

  // Slab kt is multiplied from stage kt % kStages while slab kt + kAhead is
  // copied into stage (kt + kAhead) % kStages. With one slab ahead, nothing is
  // in flight behind the slab waited for, so the wait is a full drain and the
  // copy past the last slab is simply skipped.
  static_assert(kAhead == 1, "wait counts below assume one slab ahead");
  copy_slab(0, 0);
  wait_copies_barrier<0>();
  for (int kt = 0; kt < nk; ++kt) {
    const int stage = kt & 1;
    if (kt + 1 < nk) copy_slab(kt + 1, stage ^ 1);
    const v4u* la = lds[stage];
    const v4u* lb = lds[stage] + kAChunks;
    const int c_valid = kt + 1 < nk ? 8 : c_last;
    // Four K16 steps; the fragments of step s+1 are read while step s multiplies.
    Frags f0, f1;
    read_frags(f0, la, lb, 0, wm, wn, lane, c_valid);
    read_frags(f1, la, lb, 1, wm, wn, lane, c_valid);
    mma_step<E>(acc, f0);
    read_frags(f0, la, lb, 2, wm, wn, lane, c_valid);
    mma_step<E>(acc, f1);
    read_frags(f1, la, lb, 3, wm, wn, lane, c_valid);
    mma_step<E>(acc, f0);
    mma_step<E>(acc, f1);
    wait_copies_barrier<0>();
  }
  // After the final drain no copy is in flight and every LDS read has returned:
  // the epilogue may use LDS as scratch.
  epi.tile(acc, m0, n0, wm, wn, lane, reinterpret_cast<void*>(&lds[0][0]));
  epi.finish(mt, n0, wm, wn, lane, reinterpret_cast<void*>(&lds[0][0]));
}

}  // namespace sao
