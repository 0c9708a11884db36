// MFMA tile engine for the LM-head contractions on gfx950.
//
//   C[m][n] = sum_k A[m][k] * B[n][k]      (fp32 accumulation)
//
// A workgroup of 256 threads (4 waves as 2 x 2) owns a 256 x 128 tile of C;
// each wave owns 128 x 64 as 4 x 2 MFMA 32x32 blocks held in 128 accumulator
// registers per lane. K advances in slabs of 128 bytes per row (64 bf16 or 32
// fp32 elements), double-buffered in LDS (2 stages x (32 KB of A + 16 KB of B)).
//
// Each operand is stored either K-contiguous ([mn][k], row stride ld) or
// MN-contiguous ([k][mn], row stride ld). LDS always holds [mn][k] rows of
// eight 16-byte chunks with chunk c of row r at position c ^ (r & 7), so that
// the 16-byte fragment reads of eight consecutive lanes touch all 32 banks.
// MN-contiguous operands are transposed in registers (8 x 8 bf16 or 4 x 4 fp32
// blocks) between the global load and the LDS store.
//
// Accumulator layout of v_mfma_f32_32x32x{16_bf16,2_f32} (block of 32 x 32):
// lane l, register r holds row (r & 3) + 8 * (r >> 2) + 4 * (l >> 5), column l & 31.
// Both operands feed chunk (2s + (l >> 5)) of the slab at step s, so each lane
// contributes the same k indices to A and B and the product is exact for any
// hardware ordering of k inside the instruction.
//
// Tile raster: blocks are dispatched round-robin over the 8 XCDs (block b runs
// on XCD b % 8). Every 256 consecutive blocks form one "wave" covering
// (8 * SN) N-tiles x (32 / SN) M-groups; the 32 blocks of one XCD take SN
// N-tiles x (32/SN) M-groups, so blocks sharing an XCD's L2 share operand
// panels, and all XCDs work on the same M-groups at once.
#pragma once

#include "common.hpp"

namespace sao {

constexpr int kBM = 256;                        // rows of A per tile
constexpr int kBN = 128;                        // rows of B per tile
constexpr int kMI = 4;                          // 32-row MFMA blocks per wave along M
constexpr int kNI = 2;                          // 32-column MFMA blocks per wave along N
constexpr int kThreads = 256;
constexpr int kRowChunks = 8;                   // 16-byte chunks per LDS row (128 bytes of K)
constexpr int kAChunks = kBM * kRowChunks;      // 32 KB
constexpr int kBChunks = kBN * kRowChunks;      // 16 KB
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
  int m_per_wg;            // consecutive M tiles one workgroup walks (N tile fixed)
  int m_groups;            // ceil(m_tiles / m_per_wg)
  int sn;                  // N tiles per XCD per raster wave (1, 2 or 4)
};

// Number of 256-block raster waves times 256.
inline int gemm_grid(const GemmShape& s) {
  const int nw = (s.n_tiles + 8 * s.sn - 1) / (8 * s.sn);
  const int sm = 32 / s.sn;
  const int mw = (s.m_groups + sm - 1) / sm;
  return nw * mw * 256;
}

inline int pick_sn(int n_tiles) {
  if (n_tiles % 32 == 0 || n_tiles > 96) return 4;
  if (n_tiles % 16 == 0) return 2;
  return 1;
}

template <class E>
struct Mma;

template <>
struct Mma<BF16> {
  __device__ __forceinline__ static void run(f32x16_t& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};

template <>
struct Mma<F32> {
  __device__ __forceinline__ static void run(f32x16_t& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  }
};

__device__ __forceinline__ uint4 zero4() { return make_uint4(0u, 0u, 0u, 0u); }

// Transpose of an 8 x 8 block of 16-bit values held as 8 rows of 16 bytes.
__device__ __forceinline__ void transpose8x8_b16(const uint4 (&in)[8], uint4 (&out)[8]) {
  const uint32_t* r[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = reinterpret_cast<const uint32_t*>(&in[j]);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t w[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t lo = r[2 * d][i >> 1];
      const uint32_t hi = r[2 * d + 1][i >> 1];
      w[d] = (i & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    out[i] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// Transpose of a 4 x 4 block of 32-bit values held as 4 rows of 16 bytes.
__device__ __forceinline__ void transpose4x4_b32(const uint4 (&in)[4], uint4 (&out)[4]) {
  out[0] = make_uint4(in[0].x, in[1].x, in[2].x, in[3].x);
  out[1] = make_uint4(in[0].y, in[1].y, in[2].y, in[3].y);
  out[2] = make_uint4(in[0].z, in[1].z, in[2].z, in[3].z);
  out[3] = make_uint4(in[0].w, in[1].w, in[2].w, in[3].w);
}

// Staging registers for one operand tile of R rows: 16-byte chunks per thread.
// K-contiguous tiles spread R * 8 chunks over 256 threads; MN-contiguous tiles
// give each thread whole kPerChunk x kPerChunk blocks.
template <class E, bool KC, int R>
constexpr int stage_chunks() {
  return KC ? R / 32 : ((R / E::kPerChunk + 31) / 32) * E::kPerChunk;
}

template <int N>
struct Stage {
  uint4 v[N];
};

// Global -> registers for one R-row operand tile at (mn0, k0), K-contiguous layout.
template <class E, int R>
__device__ __forceinline__ void load_kc(Stage<R / 32>& st, const typename E::storage* base, int64_t ld,
                                        int64_t mn0, int64_t mn_valid, int64_t k0, int64_t k_valid,
                                        int tid) {
  const int c = tid & 7;
  const int64_t kk = k0 + c * E::kPerChunk;
  const bool kin = kk < k_valid;
#pragma unroll
  for (int i = 0; i < R / 32; ++i) {
    int64_t row = mn0 + i * 32 + (tid >> 3);
    row = row < mn_valid ? row : mn_valid - 1;
    const uint4* p = reinterpret_cast<const uint4*>(base + row * ld + kk);
    st.v[i] = kin ? *p : zero4();
  }
}

template <int R>
__device__ __forceinline__ void store_kc(const Stage<R / 32>& st, uint4* lds, int tid) {
  const int c = tid & 7;
#pragma unroll
  for (int i = 0; i < R / 32; ++i) {
    const int row = i * 32 + (tid >> 3);
    lds[row * kRowChunks + (c ^ (row & 7))] = st.v[i];
  }
}

// Global -> registers for one R-row operand tile at (mn0, k0), MN-contiguous layout
// ([k][mn], row stride ld). The tile is 8 K chunks x R / kPerChunk MN chunks of
// kPerChunk x kPerChunk blocks; thread tid owns K chunk (tid & 7) and MN chunks
// (tid >> 3) + 32 j, each loaded as kPerChunk 16-byte rows. Rows k >= k_valid
// read as zero; MN chunks past mn_valid are clamped to the last valid chunk
// (their results are unused). Threads without a block (R = 128, bf16) idle.
template <class E, int R>
__device__ __forceinline__ void load_mc(Stage<stage_chunks<E, false, R>()>& st, const typename E::storage* base, int64_t ld,
                                        int64_t mn0, int64_t mn_valid, int64_t k0, int64_t k_valid,
                                        int tid) {
  constexpr int P = E::kPerChunk;
  constexpr int NMC = R / P;                         // MN chunks in the tile
  constexpr int NB = (NMC + 31) / 32;                // blocks per thread
  const int kc = tid & 7;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int mc = (tid >> 3) + 32 * j;
    if (NMC < 32 && mc >= NMC) break;
    int64_t mn = mn0 + mc * P;
    mn = mn < mn_valid ? mn : ((mn_valid - 1) / P) * P;
#pragma unroll
    for (int e = 0; e < P; ++e) {
      const int64_t kk = k0 + kc * P + e;
      const uint4* p = reinterpret_cast<const uint4*>(base + kk * ld + mn);
      st.v[j * P + e] = kk < k_valid ? *p : zero4();
    }
  }
}

template <class E, int R>
__device__ __forceinline__ void store_mc(const Stage<stage_chunks<E, false, R>()>& st, uint4* lds, int tid) {
  constexpr int P = E::kPerChunk;
  constexpr int NMC = R / P;
  constexpr int NB = (NMC + 31) / 32;
  const int kc = tid & 7;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int mc = (tid >> 3) + 32 * j;
    if (NMC < 32 && mc >= NMC) break;
    if constexpr (P == 8) {
      uint4 in[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) in[e] = st.v[e];
      uint4 out[8];
      transpose8x8_b16(in, out);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int row = mc * 8 + i;
        lds[row * kRowChunks + (kc ^ (row & 7))] = out[i];
      }
    } else {
      uint4 in[4] = {st.v[j * 4 + 0], st.v[j * 4 + 1], st.v[j * 4 + 2], st.v[j * 4 + 3]};
      uint4 out[4];
      transpose4x4_b32(in, out);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = mc * 4 + i;
        lds[row * kRowChunks + (kc ^ (row & 7))] = out[i];
      }
    }
  }
}

template <class E, bool KC, int R>
__device__ __forceinline__ void load_op(Stage<stage_chunks<E, KC, R>()>& st, const void* base, int64_t ld, int64_t mn0,
                                        int64_t mn_valid, int64_t k0, int64_t k_valid, int tid) {
  const auto* p = static_cast<const typename E::storage*>(base);
  if constexpr (KC)
    load_kc<E, R>(st, p, ld, mn0, mn_valid, k0, k_valid, tid);
  else
    load_mc<E, R>(st, p, ld, mn0, mn_valid, k0, k_valid, tid);
}

template <class E, bool KC, int R>
__device__ __forceinline__ void store_op(const Stage<stage_chunks<E, KC, R>()>& st, uint4* lds, int tid) {
  if constexpr (KC)
    store_kc<R>(st, lds, tid);
  else
    store_mc<E, R>(st, lds, tid);
}

// One 128-byte K slab of MFMA work for this wave from LDS.
template <class E>
__device__ __forceinline__ void mma_slab(f32x16_t (&acc)[kMI][kNI], const uint4* la, const uint4* lb,
                                         int wm, int wn, int lane) {
  const int r32 = lane & 31;
  const int hf = lane >> 5;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int c = 2 * s + hf;
    uint4 fa[kMI], fb[kNI];
#pragma unroll
    for (int i = 0; i < kMI; ++i) {
      const int ra = wm * (kBM / 2) + i * 32 + r32;
      fa[i] = la[ra * kRowChunks + (c ^ (ra & 7))];
    }
#pragma unroll
    for (int j = 0; j < kNI; ++j) {
      const int rb = wn * (kBN / 2) + j * 32 + r32;
      fb[j] = lb[rb * kRowChunks + (c ^ (rb & 7))];
    }
#pragma unroll
    for (int i = 0; i < kMI; ++i)
#pragma unroll
      for (int j = 0; j < kNI; ++j) Mma<E>::run(acc[i][j], fa[i], fb[j]);
  }
}

// Row index inside the 256-row tile of accumulator (mi, register r) for this lane.
__device__ __forceinline__ int acc_row(int wm, int mi, int r, int lane) {
  return wm * (kBM / 2) + mi * 32 + (r & 3) + 8 * (r >> 2) + 4 * (lane >> 5);
}
__device__ __forceinline__ int acc_col(int wn, int ni, int lane) { return wn * (kBN / 2) + ni * 32 + (lane & 31); }

// The generic kernel body. Epi provides:
//   begin(n0, wm, wn, lane)          once, before the first tile
//   tile(acc, m0, n0, wm, wn, lane)  after each finished 256 x 256 tile
//   finish(mg, n0, wm, wn, lane, lds) once, after the last tile (LDS is free)
template <class E, bool AKC, bool BKC, class Epi>
__device__ __forceinline__ void gemm_body(const GemmShape& s, Epi& epi, uint4 (*lds)[kStageChunks]) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1;
  const int wn = wave & 1;

  // Raster: block -> (N tile, M group).
  const int b = blockIdx.x;
  const int sn = s.sn;
  const int sm = 32 / sn;
  const int nw = (s.n_tiles + 8 * sn - 1) / (8 * sn);
  const int w = b >> 8;
  const int xcd = b & 7;
  const int slot = (b >> 3) & 31;
  const int n_tile = (w % nw) * 8 * sn + xcd * sn + (slot % sn);
  const int mg = (w / nw) * sm + slot / sn;

  const int64_t n_valid = s.n_dev ? static_cast<int64_t>(*s.n_dev) : s.n;
  const int64_t m_valid = s.m_dev ? static_cast<int64_t>(*s.m_dev) : s.m;
  const int64_t k_valid = s.k_dev ? static_cast<int64_t>(*s.k_dev) : s.k;
  if (n_tile >= s.n_tiles || mg >= s.m_groups) return;
  const int64_t n0 = static_cast<int64_t>(n_tile) * kBN;
  if (n0 >= n_valid || k_valid <= 0 || m_valid <= 0) return;
  const int m_tiles_live = static_cast<int>((m_valid + kBM - 1) / kBM);
  const int mt_begin = mg * s.m_per_wg;
  const int mt_end = min(mt_begin + s.m_per_wg, min(s.m_tiles, m_tiles_live));
  if (mt_begin >= mt_end) return;

  constexpr int kSlab = 8 * E::kPerChunk;  // K elements per slab
  const int nk = static_cast<int>((k_valid + kSlab - 1) / kSlab);
  const int total = (mt_end - mt_begin) * nk;

  epi.begin(n0, wm, wn, lane);

  f32x16_t acc[kMI][kNI];
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < kNI; ++j) acc[i][j] = f32x16_t{};

  Stage<stage_chunks<E, AKC, kBM>()> sa;
  Stage<stage_chunks<E, BKC, kBN>()> sb;
  load_op<E, AKC, kBM>(sa, s.a, s.lda, static_cast<int64_t>(mt_begin) * kBM, m_valid, 0, k_valid, tid);
  load_op<E, BKC, kBN>(sb, s.b, s.ldb, n0, n_valid, 0, k_valid, tid);
  store_op<E, AKC, kBM>(sa, lds[0], tid);
  store_op<E, BKC, kBN>(sb, lds[0] + kAChunks, tid);
  __syncthreads();

  int f = 0;
  for (int mt = mt_begin; mt < mt_end; ++mt) {
    for (int kt = 0; kt < nk; ++kt, ++f) {
      const int buf = f & 1;
      const bool last_k = kt + 1 == nk;
      const bool more = (f + 1) < total;
      if (more) {
        const int nmt = last_k ? mt + 1 : mt;
        const int nkt = last_k ? 0 : kt + 1;
        load_op<E, AKC, kBM>(sa, s.a, s.lda, static_cast<int64_t>(nmt) * kBM, m_valid,
                        static_cast<int64_t>(nkt) * kSlab, k_valid, tid);
        load_op<E, BKC, kBN>(sb, s.b, s.ldb, n0, n_valid, static_cast<int64_t>(nkt) * kSlab, k_valid, tid);
      }
      mma_slab<E>(acc, lds[buf], lds[buf] + kAChunks, wm, wn, lane);
      if (more) {
        store_op<E, AKC, kBM>(sa, lds[buf ^ 1], tid);
        store_op<E, BKC, kBN>(sb, lds[buf ^ 1] + kAChunks, tid);
      }
      __syncthreads();
    }
    epi.tile(acc, static_cast<int64_t>(mt) * kBM, n0, wm, wn, lane);
#pragma unroll
    for (int i = 0; i < kMI; ++i)
#pragma unroll
      for (int j = 0; j < kNI; ++j) acc[i][j] = f32x16_t{};
  }
  epi.finish(mg, n0, wm, wn, lane, reinterpret_cast<void*>(&lds[0][0]));
}

}  // namespace sao
