// MFMA tile engine for the LM-head contractions on gfx950.
//
//   C[m][n] = sum_k A[m][k] * B[n][k]      (fp32 accumulation)
//
// A workgroup of 256 threads (4 waves as 2 x 2) owns a 256 x 256 tile of C;
// each wave owns 128 x 128 as 4 x 4 MFMA 32x32 blocks held in 256 accumulator
// registers per lane. K advances in slabs of kRowChunks x 16 bytes per row (64
// bf16 or 32 fp32 elements) through an LDS ring of kStages x (32 KB of A + 32 KB
// of B). Slabs are copied global -> LDS directly (global_load_lds_dwordx4: no
// staging registers, no LDS store instructions), kStages - 1 slabs ahead of the
// MFMAs.
//
// Each operand is stored either K-major ([mn][k], row stride ld) or MN-major
// ([k][mn], row stride ld), chosen at compile time. A K-major slab sits in LDS
// as [mn][k] rows of kRowChunks 16-byte chunks, chunk c of row r at position
// swz(r, c), so that the 16-byte fragment reads of sixteen consecutive lanes
// touch all 64 banks. An MN-major slab sits as [k][mn] rows of 256 elements,
// chunk c of row k at c ^ (4 (k & 3)); bf16 fragments come from it through
// gfx950's transposing LDS read (ds_read_b64_tr_b16: within each 16 lanes,
// lane j names 4 elements of row j >> 2 and receives column j of the 4 x 16
// block that the group names), two reads per 8-element fragment, and the
// XOR keeps the 32 lanes of each read on distinct banks.
//
// Issue schedule. Each SIMD runs one wave of the workgroup and a wave issues
// in order, so anything issued in a burst between MFMAs leaves the MFMA pipe
// idle. The fragments of K step s+1 are therefore read one per MFMA over the
// first half of step s, in the order step s+1 uses them, and the copies of a
// slab go one after every other MFMA: half in the last step of the slab two
// before it (right after the barrier that frees their stage), half in step 0
// of the slab just before it. The workgroup barrier of a slab sits before its
// last K step, so the first fragments of the next slab are read while that
// step multiplies. (Measured at the LM-head forward shape: bursts of reads and
// copies cost 103k cycles per tile against 65.5k of MFMA work, this schedule
// 81k. Deeper rings of shorter slabs measured slower: the extra barriers cost
// more than the added copy slack gains.)
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
// (SN x 256/SN), so an M-tile's rows are fetched by one XCD only. The split
// dimension is dealt out to the XCDs in turn (XCD x takes tiles x, x + 8, ...),
// so that when only part of it holds valid rows (a device-side count below the
// host bound) every XCD still gets its share of the work. In N-split mode the
// XCD-to-column assignment rotates by one XCD from one M group to the next.
// (Measured: with 162 N tiles the forward ran 12 % faster rotated; rotating
// only the last, partial N group gained nothing, so this is not the tail's
// balance alone. With 181 N tiles rotation costs about 0.5 %.) M-split keeps
// the assignment fixed, so that each XCD keeps streaming its own M tiles.
#pragma once

#include <type_traits>
#include <utility>

#include "common.hpp"

namespace sao {

constexpr int kBM = 256;                        // rows of A per tile
constexpr int kBN = 256;                        // rows of B per tile
constexpr int kMI = 4;                          // 32-row MFMA blocks per wave along M
constexpr int kNI = 4;                          // 32-column MFMA blocks per wave along N
constexpr int kThreads = 256;                   // 4 waves: 2 along M x 2 along N, one per SIMD
constexpr int kWavesN = 2;
constexpr int kRowChunks = 8;                   // 16-byte chunks per LDS row (128 bytes of K)
constexpr int kAChunks = kBM * kRowChunks;      // 32 KB
constexpr int kBChunks = kBN * kRowChunks;      // 32 KB
constexpr int kStages = 2;                      // LDS ring depth
constexpr int kRowsPerCopy = 64 / kRowChunks;   // tile rows filled by one wave-wide 1 KB copy
constexpr int kSteps = kRowChunks / 2;          // MFMA K steps per slab (two chunks each)
constexpr int kRowsPerLine = 16 / kRowChunks;   // tile rows per 256-byte line of the 64 banks
static_assert(kSteps % 2 == 0, "the next slab's first step lands in f0");
constexpr int kStageChunks = kAChunks + kBChunks;
// Of the copies per wave of one slab, kCopyNow are issued in the last K step
// of the slab two before it and the rest in step 0 of the slab just before it.
constexpr int kCopyNow = 8;

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
  int64_t k_split;         // > 0: K is cut into pieces of this length (a multiple of 64),
                           // piece blockIdx.y per workgroup; the epilogue keeps them apart
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

// N-split: SN so that 8 SN N-tiles fill the N range with little waste. (For
// the backward's logit recompute at 256 token tiles, SN 8 measured 0.8 % faster
// than 4 and SN 2 1.7 % slower; at 128 token tiles SN 8 was 1.8 % slower.)
inline int pick_sn(int n_tiles) {
  if (n_tiles > 128) return 8;
  if (n_tiles % 32 == 0 || n_tiles > 96) return 4;
  if (n_tiles % 16 == 0) return 2;
  return 1;
}

// Launches with at most this many N tiles (host bound) use the M-split raster.
constexpr int kMsplitMaxNTiles = 64;

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
// 16-byte access per cycle across 64 banks (one 256-byte line, kRowsPerLine
// rows), so the 16 consecutive rows read by lanes 0-15 at one logical chunk
// must land on 16 distinct (row within line, chunk) pairs: XOR with the line
// index modulo kRowChunks does that.
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r / kRowsPerLine) % kRowChunks); }

// A wave-uniform value as a scalar (the builtin yields a signed int: going
// through uint32_t keeps a widened address from being sign-extended).
__device__ __forceinline__ uint32_t uniform_u32(uint32_t x) {
  return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(x)));
}
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint64_t lo = uniform_u32(static_cast<uint32_t>(v));
  const uint64_t hi = uniform_u32(static_cast<uint32_t>(v >> 32));
  return reinterpret_cast<const void*>((hi << 32) | lo);
}

// Direct copy of 16 bytes per lane from global memory (uniform base `g` plus the
// lane's byte offset `off`) into LDS: lane l writes LDS bytes [m0 + 16 l, +16),
// m0 being the wave-uniform LDS byte address lds_base + lds_off (summed straight
// into m0). Issued as inline assembly so that the compiler does not insert its
// conservative full waits before every LDS read; completion is tracked with
// explicit vmcnt waits.
__device__ __forceinline__ void dma16(const void* g, uint32_t off, uint32_t lds_base, uint32_t lds_off) {
  asm volatile("s_add_u32 m0, %2, %3\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(g), "s"(lds_base),
               "s"(lds_off)
               : "memory", "m0", "scc");
}

// This wave's copies except the N most recent have landed in LDS, its LDS
// reads have returned, then the workgroup barrier: afterwards every wave's
// copies of the awaited slab are visible and the stage read before is free.
// Copies complete in issue order, so the N most recent are the later slabs.
template <int N>
__device__ __forceinline__ void wait_copies_barrier() {
  if constexpr (N == 0)
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  else
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(N) : "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// The same with N = PerSlab * pending for a wave-uniform `pending` in
// [0, kStages - 1] (the count must be an immediate).
template <int PerSlab, int P = kStages - 1>
__device__ __forceinline__ void wait_slabs_barrier(int pending) {
  if constexpr (P == 0) {
    wait_copies_barrier<0>();
  } else {
    if (pending >= P)
      wait_copies_barrier<PerSlab * P>();
    else
      wait_slabs_barrier<PerSlab, P - 1>(pending);
  }
}

// Instruction order is pinned where it matters: the compiler would otherwise
// defer the LDS reads of the next K step behind the MFMAs of this one and then
// wait for them, exposing the LDS latency once per step.
__device__ __forceinline__ void pin_order() { __builtin_amdgcn_sched_barrier(0); }

// Fragments of one K16 step (bf16; K8 for fp32): kMI rows of A, kNI rows of B.
struct Frags {
  v4u a[kMI];
  v4u b[kNI];
};

// K-major fragment i (rows wave_row0 + 32 i ..) of one operand for K step s.
// Rows read by a lane differ by multiples of 32, which leaves the line index
// modulo kRowChunks and hence the swizzle unchanged: one LDS address per step,
// the blocks at immediate offsets. Chunks past K hold zeros (written by the
// copy of the last slab), so no fragment needs masking.
__device__ __forceinline__ v4u read_frag_k(const v4u* l, int s, int wave_row0, int i, int lane) {
  const int r32 = lane & 31;
  const int c = 2 * s + (lane >> 5);
  return l[(wave_row0 + r32) * kRowChunks + swz(r32, c) + i * 32 * kRowChunks];
}

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

// MN-major slab geometry for element type E: rows of 256 elements.
template <class E>
struct MnSlab {
  static constexpr int kRowBytes = 256 * static_cast<int>(sizeof(typename E::storage));
  static constexpr int kChunksPerRow = kRowBytes / 16;
  static constexpr int kRows = kRowChunks * E::kPerChunk;        // K per slab
  static constexpr int kRowsPerCopy = 1024 / kRowBytes;           // rows filled by one 1 KB copy
  static_assert(kRows * kRowBytes == kAChunks * 16, "an MN-major slab fills one operand stage");
};
__device__ __forceinline__ int mn_swz(int k, int c) { return c ^ (4 * (k & 3)); }

// MN-major fragment i of one operand for K step s (same k <-> lane mapping as
// the K-major path: lane half h holds the k chunk 2 s + h, element e at k offset e).
template <class E>
__device__ __forceinline__ v4u read_frag_mn(const v4u* l, int s, int wave_row0, int i, int lane) {
  using G = MnSlab<E>;
  const char* base = reinterpret_cast<const char*>(l);
  const int h = lane >> 5;
  if constexpr (sizeof(typename E::storage) == 2) {
    // Lane j of a 16-lane group names row k0 + (j >> 2), columns m0 + 4 (j & 3) .. +3,
    // and receives column m0 + j of rows k0 .. k0+3; two reads give rows k0 .. k0+7.
    const int j = lane & 15;
    const int k = 8 * (2 * s + h) + (j >> 2);
    const int m = wave_row0 + 32 * i + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
    const int off = k * G::kRowBytes + mn_swz(k, m >> 3) * 16 + (m & 7) * 2;
    const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(base + off));
    const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(base + off + 4 * G::kRowBytes));
    const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
    return v4u{a.x, a.y, b.x, b.y};
  } else {
    // fp32: element e of the chunk is row 4 (2 s + h) + e of column wave_row0 + 32 i + (lane & 31).
    const int m = wave_row0 + 32 * i + (lane & 31);
    uint32_t x[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = 4 * (2 * s + h) + e;
      x[e] = *reinterpret_cast<const uint32_t*>(base + k * G::kRowBytes + mn_swz(k, m >> 2) * 16 + (m & 3) * 4);
    }
    return v4u{x[0], x[1], x[2], x[3]};
  }
}

// Fragment idx (0 .. kMI + kNI - 1) of K step s in the order in which the
// MFMAs of a step first use them: A0, B0, B1, .., B(kNI-1), A1, .., A(kMI-1).
template <class E, bool AMn, bool BMn>
__device__ __forceinline__ void read_one(Frags& f, int idx, const v4u* la, const v4u* lb, int s, int wm, int wn,
                                         int lane) {
  const bool is_a = idx == 0 || idx > kNI;
  const int i = idx == 0 ? 0 : idx - kNI;
  if (is_a) {
    if constexpr (AMn)
      f.a[i] = read_frag_mn<E>(la, s, wm * (kBM / 2), i, lane);
    else
      f.a[i] = read_frag_k(la, s, wm * (kBM / 2), i, lane);
  } else {
    if constexpr (BMn)
      f.b[idx - 1] = read_frag_mn<E>(lb, s, wn * (kBN / kWavesN), idx - 1, lane);
    else
      f.b[idx - 1] = read_frag_k(lb, s, wn * (kBN / kWavesN), idx - 1, lane);
  }
}

template <class E, bool AMn, bool BMn>
__device__ __forceinline__ void read_frags(Frags& f, const v4u* la, const v4u* lb, int s, int wm, int wn,
                                           int lane) {
#pragma unroll
  for (int idx = 0; idx < kMI + kNI; ++idx) {
    read_one<E, AMn, BMn>(f, idx, la, lb, s, wm, wn, lane);
    pin_order();  // in the same order as the loop reads them, so waits agree
  }
}

// One K step of one wave: the kMI x kNI MFMAs of `cur`, with the fragments of
// the next step (read into `nxt` from la / lb) and the hook's copies placed
// between them. A wave issues in order and each SIMD runs one wave, so the
// MFMA pipe idles while the wave issues a burst of other instructions; the
// reads therefore go one after every kReadEvery MFMAs, in the order in which
// the next step uses them, and the hook may add a copy after any MFMA.
constexpr int kReadEvery = 1;
static_assert((kMI + kNI) * kReadEvery <= kMI * kNI, "all reads fit in one step");
template <class E, bool AMn, bool BMn, class Hook>
__device__ __forceinline__ void mma_step_mix(f32x16_t (&acc)[kMI][kNI], const Frags& cur, Frags& nxt,
                                             const v4u* la, const v4u* lb, int s_next, int wm, int wn,
                                             int lane, Hook&& hook) {
  // The MFMAs run in snake order (even rows of blocks left to right, odd rows
  // right to left), so the B fragment stays the same across each row change:
  // fewer operand bits switch between consecutive MFMAs, which costs less power.
  // The fragments' first uses keep the read order above.
#pragma unroll
  for (int t = 0; t < kMI * kNI; ++t) {
    const int mi = t / kNI;
    const int ni = mi % 2 == 0 ? t % kNI : kNI - 1 - t % kNI;
    Mma<E>::run(acc[mi][ni], cur.a[mi], cur.b[ni]);
    pin_order();
    if (t % kReadEvery == kReadEvery - 1 && t / kReadEvery < kMI + kNI)
      read_one<E, AMn, BMn>(nxt, t / kReadEvery, la, lb, s_next, wm, wn, lane);
    hook(t);
    pin_order();
  }
}

// LDS writes of this thread are complete, then the workgroup barrier. Unlike
// __syncthreads() this does not wait for outstanding global loads, which keeps
// the next slab's prefetch in flight across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One accumulator element, read out of its AGPR at this point of the program.
// Left to itself the compiler moves all 256 accumulators to VGPRs as soon as the
// K loop ends, which leaves no room for anything else in an epilogue and spills;
// reading each element where it is used keeps the epilogue's VGPRs few.
__device__ __forceinline__ float acc_read(float x) {
  float r;
  asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(r) : "a"(x));
  return r;
}

// Row index inside the 256-row tile of accumulator (mi, register r) for this lane.
__device__ __forceinline__ int acc_row(int wm, int mi, int r, int lane) {
  return wm * (kBM / 2) + mi * 32 + (r & 3) + 8 * (r >> 2) + 4 * (lane >> 5);
}
__device__ __forceinline__ int acc_col(int wn, int ni, int lane) {
  return wn * (kBN / kWavesN) + ni * 32 + (lane & 31);
}

// Optional timeline marks of an epilogue (a measurement hook): mark(0) after the
// prologue (the first slab has landed), mark(1) after the K loop.
template <class Epi, class = void>
struct HasMark : std::false_type {};
template <class Epi>
struct HasMark<Epi, std::void_t<decltype(std::declval<Epi&>().mark(0))>> : std::true_type {};
template <class Epi>
__device__ __forceinline__ void epi_mark(Epi& epi, int phase) {
  if constexpr (HasMark<Epi>::value) epi.mark(phase);
}

template <class E, bool AMn, bool BMn, class Epi>
__device__ __forceinline__ void gemm_tile(const GemmShape& s, Epi& epi, v4u (*lds)[kStageChunks], int mt,
                                          int n_tile);

// The generic kernel body: one 256 x 256 tile per workgroup. Epi provides:
//   begin(n0, wm, wn, lane)                 before the K loop
//   tile(acc, m0, n0, wm, wn, lane, lds)    after it (LDS is free)
//   finish(mt, n0, wm, wn, lane, lds)  last (LDS is free)
// AMn / BMn select the MN-major layout for A / B.
template <class E, bool AMn, bool BMn, class Epi>
__device__ __forceinline__ void gemm_body(const GemmShape& s, Epi& epi, v4u (*lds)[kStageChunks]) {
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
    mt = (w / nw) * (256 / sn) + (slot / sn) * 8 + xcd;
  } else {
    n_tile = (w % nw) * 8 * sn + (slot % sn) * 8 + (xcd + w / nw) % 8;
    mt = (w / nw) * (32 / sn) + slot / sn;
  }
  gemm_tile<E, AMn, BMn>(s, epi, lds, mt, n_tile);
}

// Tile (mt, n_tile) of the product, K piece blockIdx.y; nothing if the tile
// lies past the valid rows.
template <class E, bool AMn, bool BMn, class Epi>
__device__ __forceinline__ void gemm_tile(const GemmShape& s, Epi& epi, v4u (*lds)[kStageChunks], int mt,
                                          int n_tile) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = static_cast<int>(uniform_u32(static_cast<uint32_t>(tid >> 6)));  // keeps copy addresses scalar
  const int wm = wave / kWavesN;
  const int wn = wave % kWavesN;

  const int64_t n_valid = s.n_dev ? static_cast<int64_t>(*s.n_dev) : s.n;
  const int64_t m_valid = s.m_dev ? static_cast<int64_t>(*s.m_dev) : s.m;
  int64_t k_valid = s.k_dev ? static_cast<int64_t>(*s.k_dev) : s.k;
  int64_t k0 = 0;  // first K index of this workgroup's piece
  if (s.k_split > 0) {
    k0 = static_cast<int64_t>(blockIdx.y) * s.k_split;
    k_valid = k_valid - k0 < s.k_split ? k_valid - k0 : s.k_split;
  }
  if (n_tile >= s.n_tiles || mt >= s.m_tiles) return;
  const int64_t n0 = static_cast<int64_t>(n_tile) * kBN;
  const int64_t m0 = static_cast<int64_t>(mt) * kBM;
  if (n0 >= n_valid || m0 >= m_valid || k_valid <= 0) return;

  constexpr int P = E::kPerChunk;
  const int64_t k_chunks = (k_valid + P - 1) / P;          // valid 16-byte chunks per row
  const int nk = static_cast<int>((k_chunks + kRowChunks - 1) / kRowChunks);  // slabs

  epi.begin(n0, wm, wn, lane);

  f32x16_t acc[kMI][kNI];
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < kNI; ++j) acc[i][j] = f32x16_t{};

  const int esz = static_cast<int>(sizeof(typename E::storage));
  // The scalar bases point at the tile's first row (K-major) or column
  // (MN-major) of the K piece, so that a lane's 32-bit offset spans one tile
  // of rows or one slab of k rows, whatever the operand's size.
  const char* a_base = static_cast<const char*>(s.a) + (AMn ? k0 * s.lda + m0 : k0 + m0 * s.lda) * esz;
  const char* b_base = static_cast<const char*>(s.b) + (BMn ? k0 * s.ldb + n0 : k0 + n0 * s.ldb) * esz;
  using G = MnSlab<E>;
  // Every 1 KB copy instruction of a wave fills 64 consecutive LDS chunks (lane l
  // writes chunk l). K-major: copy q covers kRowsPerCopy tile rows from
  // (wave * Q + q) * kRowsPerCopy, lane l row + l / kRowChunks at physical chunk
  // l % kRowChunks, fetching the logical chunk swizzled there; lc[q] is that chunk
  // and off[q] the byte offset of that row and chunk in slab 0. MN-major: copy q covers G::kRowsPerCopy slab
  // rows (k) from (wave * Q + q) * G::kRowsPerCopy, lane l row + l / G::kChunksPerRow
  // at physical chunk l % G::kChunksPerRow, fetching the logical column chunk
  // mn_swz maps there; lc[q] is the slab row and off[q] the byte offset of that
  // row and column in slab 0. Offsets are relative to the tile's base. Rows
  // (K-major) or columns (MN-major) past the valid range read the last valid
  // one; their results are never stored.
  constexpr int QA = kAChunks / 64 / (kThreads / 64);  // copies per wave per A slab
  constexpr int QB = kBChunks / 64 / (kThreads / 64);  // copies per wave per B slab
  constexpr int kCopiesPerSlab = QA + QB;
  uint32_t offa[QA], offb[QB];
  int lca[QA], lcb[QB];
  auto setup = [&](auto mn_major, int Q, int q, int64_t row0, int64_t valid, int64_t ld, uint32_t& off, int& lc) {
    if constexpr (decltype(mn_major)::value) {
      const int k = (wave * Q + q) * G::kRowsPerCopy + lane / G::kChunksPerRow;
      const int c = mn_swz(k, lane % G::kChunksPerRow);
      int64_t col = static_cast<int64_t>(c) * P;                     // from the tile's first column
      if (row0 + col >= valid) col = (valid - 1) / P * P - row0;    // row0 is a multiple of P
      lc = k;
      off = static_cast<uint32_t>((static_cast<int64_t>(k) * ld + col) * esz);
    } else {
      const int r = (wave * Q + q) * kRowsPerCopy + lane / kRowChunks;
      lc = swz(r, lane % kRowChunks);
      const int64_t row = row0 + r < valid ? r : valid - 1 - row0;  // from the tile's first row
      off = static_cast<uint32_t>(row * ld * esz + static_cast<int64_t>(lc) * P * esz);
    }
  };
#pragma unroll
  for (int q = 0; q < QA; ++q) setup(std::bool_constant<AMn>{}, QA, q, m0, m_valid, s.lda, offa[q], lca[q]);
#pragma unroll
  for (int q = 0; q < QB; ++q) setup(std::bool_constant<BMn>{}, QB, q, n0, n_valid, s.ldb, offb[q], lcb[q]);
  // Byte offset of slab kt for copy q, and whether that copy's data lies inside K.
  const int64_t slab_a = static_cast<int64_t>(G::kRows) * s.lda * esz;
  const int64_t slab_b = static_cast<int64_t>(G::kRows) * s.ldb * esz;
  const uint32_t lds0 = uniform_u32(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&lds[0][0])));
  v4u* lds_flat = &lds[0][0];
  // Scalar base address of slab kt of operand A or B (the slab's offset is
  // uniform and goes into the base; the lanes' offsets stay fixed).
  auto slab_ptr = [&](bool is_a, int kt) -> const char* {
    const bool mn = is_a ? AMn : BMn;
    const int64_t k_off = mn ? static_cast<int64_t>(kt) * (is_a ? slab_a : slab_b)
                             : static_cast<int64_t>(kt) * kRowChunks * P * esz;
    return static_cast<const char*>(uniform_ptr((is_a ? a_base : b_base) + k_off));
  };
  // Copy q of a slab whose A and B bases are ga and gb, into `stage`.
  auto copy_at = [&](int q, const char* ga, const char* gb, int stage) {
    const bool is_a = q < QA;
    const int qq = is_a ? q : q - QA;
    const int slot = (is_a ? 0 : kAChunks) + (wave * (is_a ? QA : QB) + qq) * 64;
    dma16(is_a ? ga : gb, is_a ? offa[qq] : offb[qq],
          uniform_u32(lds0 + static_cast<uint32_t>(stage * kStageChunks) * 16),
          uniform_u32(static_cast<uint32_t>(slot) * 16));
  };
  auto copy_one = [&](int q, int kt, int stage) {
    copy_at(q, q < QA ? slab_ptr(true, kt) : nullptr, q < QA ? nullptr : slab_ptr(false, kt), stage);
  };
  auto inside_k = [&](int q, int kt) -> bool {
    const bool is_a = q < QA;
    const int qq = is_a ? q : q - QA;
    const int lc = is_a ? lca[qq] : lcb[qq];
    if (is_a ? AMn : BMn) return static_cast<int64_t>(kt) * G::kRows + lc < k_valid;
    return static_cast<int64_t>(kt) * kRowChunks + lc < k_chunks;
  };
  // The last slab is partial when K ends inside it. Then lanes whose data lies
  // past K write zeros to their LDS slot instead of copying. A K-major copy
  // always keeps chunk 0 of its rows, but an MN-major one can lose all its rows:
  // its instruction is then not issued, so waits that count copies must not
  // span that slab.
  const bool tail = k_valid < static_cast<int64_t>(nk) * G::kRows;
  auto copy_slab = [&](int kt, int stage) {
    if (kt == nk - 1 && tail) {
#pragma unroll
      for (int q = 0; q < kCopiesPerSlab; ++q) {
        const bool is_a = q < QA;
        const int qq = is_a ? q : q - QA;
        const int slot = (is_a ? 0 : kAChunks) + (wave * (is_a ? QA : QB) + qq) * 64;
        if (inside_k(q, kt))
          copy_one(q, kt, stage);
        else
          lds_flat[stage * kStageChunks + slot + lane] = zero4();
      }
    } else {
#pragma unroll
      for (int q = 0; q < kCopiesPerSlab; ++q) copy_one(q, kt, stage);
    }
  };

  // Slab kt is multiplied from stage kt % kStages while slabs kt+1 .. kt+3 are
  // in flight or landed. Once every wave has read slab kt's last fragments (the
  // barrier inside iteration kt), its stage takes slab kt + kStages. Before that
  // barrier this wave's copies of slab kt+1 must have landed; the ones issued
  // after them (slabs kt+2 and kt+3, as far as they exist) may stay in flight.
  for (int j = 0; j < kStages; ++j)
    if (j < nk) copy_slab(j, j);
  {
    int pending = nk - 1 < kStages - 1 ? nk - 1 : kStages - 1;
    if (tail && nk <= kStages) pending = 0;  // the partial slab is among these copies
    wait_slabs_barrier<kCopiesPerSlab>(pending);
  }
  epi_mark(epi, 0);
  Frags f0, f1;
  read_frags<E, AMn, BMn>(f0, lds[0], lds[0] + kAChunks, 0, wm, wn, lane);
  constexpr int kCopyNext = kCopiesPerSlab - kCopyNow;
  static_assert(kCopyNow > 0 && kCopyNext > 0 && (kMI * kNI) % kCopyNow == 0 && (kMI * kNI) % kCopyNext == 0,
                "copies spread evenly over a step's MFMAs");
  // Whether the previous iteration left copies of slab kt + 1 to step 0 (a
  // wave-uniform scalar, so that the copies' guards are scalar branches).
  uint32_t carry = 0;
  // One slab. In the steady state (kSteady: 1 <= kt <= nk - 4) every copy is
  // issued, so those iterations carry no guards at all.
  auto slab = [&](int kt, auto steady) {
    constexpr bool kSteady = decltype(steady)::value;
    const int stage = kt % kStages;
    const int cstage = (kt + 1) % kStages;
    // K steps 0 .. kSteps-2 multiply f0 / f1 (even / odd steps) while reading
    // the next step's fragments from this stage. Step 0 also issues the copies
    // of slab kt + 1 that the previous iteration left over. The slab's scalar
    // bases are formed once, not per copy.
    constexpr int kEveryNext = kMI * kNI / kCopyNext;
    const char* ga1 = slab_ptr(true, kt + 1);
    const char* gb1 = slab_ptr(false, kt + 1);
#pragma unroll
    for (int st = 0; st + 1 < kSteps; ++st) {
      Frags& cur = st % 2 == 0 ? f0 : f1;
      Frags& nxt = st % 2 == 0 ? f1 : f0;
      mma_step_mix<E, AMn, BMn>(acc, cur, nxt, lds[stage], lds[stage] + kAChunks, st + 1, wm, wn, lane,
                                [&](int t) {
                                  if (st == 0 && t % kEveryNext == kEveryNext - 1 && (kSteady || carry))
                                    copy_at(kCopyNow + t / kEveryNext, ga1, gb1, cstage);
                                });
    }
    Frags& last = kSteps % 2 == 0 ? f1 : f0;
    const int kn = kt + kStages;  // the slab that refills this stage
    if (kSteady || kt + 1 < nk) {
      const int rest = nk - kt - 2;
      wait_slabs_barrier<kCopiesPerSlab>(rest < kStages - 2 ? rest : kStages - 2);
    }
    // The last step reads the next slab's first fragments (unconditionally, so
    // that the LDS wait counts agree on both paths; after the last slab it reads
    // a drained stage and the values go unused). Full slabs refill the freed
    // stage: kCopyNow copies spread over this step's MFMAs, the rest over step 0
    // of the next slab; the last slab, when K ends inside it, is copied after
    // them with its zero fill.
    const uint32_t refill = kSteady ? 1u : uniform_u32(kn < nk - 1 || (kn == nk - 1 && !tail) ? 1u : 0u);
    const char* ga2 = slab_ptr(true, kn);
    const char* gb2 = slab_ptr(false, kn);
    constexpr int kEveryNow = kMI * kNI / kCopyNow;
    mma_step_mix<E, AMn, BMn>(acc, last, f0, lds[cstage], lds[cstage] + kAChunks, 0, wm, wn, lane, [&](int t) {
      if (t % kEveryNow == kEveryNow - 1 && (kSteady || refill)) copy_at(t / kEveryNow, ga2, gb2, stage);
    });
    if (!kSteady && kn == nk - 1 && tail) copy_slab(kn, stage);
    carry = refill;
  };
  // kt = 0 (nothing carried), the steady iterations, then the last three.
  int kt = 0;
  if (nk > 0) slab(kt++, std::false_type{});
  for (; kt <= nk - 4; ++kt) slab(kt, std::true_type{});
  for (; kt < nk; ++kt) slab(kt, std::false_type{});
  // Every copy has landed (the last wait drained them); once every wave's LDS
  // reads have returned, the epilogue may use LDS as scratch.
  lds_barrier();
  epi_mark(epi, 1);
  epi.tile(acc, m0, n0, wm, wn, lane, reinterpret_cast<void*>(&lds[0][0]));
  epi.finish(mt, n0, wm, wn, lane, reinterpret_cast<void*>(&lds[0][0]));
}

}  // namespace sao
