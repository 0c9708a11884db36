// LM-head kernels of the SAO loss pass: per-token log-probs (forward) and the
// backward into hidden states and head weights, both on bf16 (or fp32) MFMA.
//
// Forward (Sec. 3.1, Eq. 1-2): rows with mask 1 are compacted, then
//   z = W_head . h_t over 256 x 256 tiles (vocabulary x tokens); each tile is
//   reduced in registers to a (max, sum exp) pair per token, so the logits never
//   leave the chip; the pairs of all vocabulary tiles are merged per token and
//   the target logit z_{t,y_t} is a separate dot product.
// Backward: rows with g != 0 are compacted (Hg); for each vocabulary block of Vc
//   rows (A) recompute z and write dz = g (onehot - exp(z - lse)) to a [T x Vc]
//   scratch, (B) dH += dz . W_block (W read MN-major), (C) dW_block += dz^T . Hg
//   (dz and Hg read MN-major), all three on MFMA.
#include "common.hpp"
#include "gemm.hpp"
#include "launch.hpp"
#include "layout.hpp"
#include "timer.hpp"
#include "../../include/sao.h"

namespace sao {

// Compacted row buffers are zero-filled up to a multiple of this many rows.
constexpr int64_t kRowPad = 256;

// ------------------------------------------------------------------------- //
// Row compaction
// ------------------------------------------------------------------------- //
__device__ __forceinline__ bool row_selected(const uint8_t* mask, const float* g, int64_t t) {
  if (mask) return mask[t] != 0;
  if (g) return g[t] != 0.0f;
  return true;
}

template <typename T>
__device__ __forceinline__ T block_sum_256(T v, T* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  return sh[0] + sh[1] + sh[2] + sh[3];
}

__global__ __launch_bounds__(256) void k_count_rows(const uint8_t* mask, const float* g, int64_t T,
                                                    int32_t* blk_counts, int32_t* zero, int n_zero) {
  __shared__ int32_t sh[4];
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i < n_zero; i += blockDim.x) zero[i] = 0;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kRowsPerCountBlock + threadIdx.x * 4;
  int32_t c = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t t = base + j;
    if (t < T && row_selected(mask, g, t)) ++c;
  }
  c = block_sum_256(c, sh);
  if (threadIdx.x == 0) blk_counts[blockIdx.x] = c;
}

// Writes idx[c] = t for the c-th selected row (ascending t), pos[t] = c or -1,
// the total to *count, and zeroes zero_a[t], zero_b[t] on unselected rows.
__global__ __launch_bounds__(256) void k_compact_rows(const uint8_t* mask, const float* g, int64_t T,
                                                      const int32_t* blk_counts, int32_t* idx,
                                                      int32_t* pos, int32_t* count, float* zero_a,
                                                      float* zero_b) {
  __shared__ int32_t sh[4];
  __shared__ int32_t s_wave[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t before = 0;
  for (int i = tid; i < static_cast<int>(blockIdx.x); i += 256) before += blk_counts[i];
  before = block_sum_256(before, sh);

  const int64_t base = static_cast<int64_t>(blockIdx.x) * kRowsPerCountBlock + tid * 4;
  bool sel[4];
  int32_t c = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t t = base + j;
    sel[j] = t < T && row_selected(mask, g, t);
    c += sel[j] ? 1 : 0;
  }
  int32_t incl = c;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int32_t o = __shfl_up(incl, d, 64);
    if (lane >= d) incl += o;
  }
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int32_t woff = 0;
  for (int w = 0; w < wave; ++w) woff += s_wave[w];
  int32_t p = before + woff + incl - c;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t t = base + j;
    if (t >= T) break;
    if (sel[j]) {
      idx[p] = static_cast<int32_t>(t);
      if (pos) pos[t] = p;
      ++p;
    } else {
      if (pos) pos[t] = -1;
      if (zero_a) zero_a[t] = 0.0f;
      if (zero_b) zero_b[t] = 0.0f;
    }
  }
  if (blockIdx.x == gridDim.x - 1 && tid == 255) *count = p;
}

// Copies the selected rows into a dense [rows][H] buffer and zero-fills up to the
// next multiple of 256 rows; gathers per-row extras alongside.
template <class E>
__global__ __launch_bounds__(256) void k_gather_rows(const typename E::storage* src, int64_t ld_src,
                                                     int64_t H, const int32_t* idx,
                                                     const int32_t* count,
                                                     typename E::storage* dst,
                                                     const int32_t* target, int32_t* y_c,
                                                     const float* g, float* g_c, const float* lse,
                                                     float* lse_c) {
  const int lane = threadIdx.x & 63;
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int64_t n = *count;
  if (c >= round_up_dev(n, kRowPad)) return;
  const int64_t chunks = H / E::kPerChunk;
  v4u* d = reinterpret_cast<v4u*>(dst + c * H);
  if (c < n) {
    const int64_t t = idx[c];
    const v4u* s = reinterpret_cast<const v4u*>(src + t * ld_src);
    for (int64_t k = lane; k < chunks; k += 64) d[k] = s[k];
    if (lane == 0) {
      if (y_c) y_c[c] = target[t];
      if (g_c) g_c[c] = g[t];
      if (lse_c) lse_c[c] = lse[t];
    }
  } else {
    for (int64_t k = lane; k < chunks; k += 64) d[k] = zero4();
    if (lane == 0) {
      if (y_c) y_c[c] = -1;
      if (g_c) g_c[c] = 0.0f;
      if (lse_c) lse_c[c] = 0.0f;
    }
  }
}

// Timeline marks of an epilogue (a measurement hook, off unless `timeline`):
// s_memtime after the prologue and after the K loop, and the tile (M tile << 32
// | N tile, -1 for none).
struct TileClock {
  bool timeline;
  uint64_t t_mark[2];
  int64_t tile_id;

  __device__ __forceinline__ void mark(int phase) {
    if (timeline) t_mark[phase] = __builtin_amdgcn_s_memtime();
  }
  __device__ __forceinline__ void start(bool on) {
    timeline = on;
    t_mark[0] = t_mark[1] = 0;
    tile_id = -1;
  }
};

// ------------------------------------------------------------------------- //
// Forward: online log-sum-exp epilogue
// ------------------------------------------------------------------------- //
// kMasked: the launch covers the last, partial vocabulary tile (rows at or past
// M read as -inf); otherwise every tile of the launch has 256 valid rows. The
// two cases are separate launches, so that each kernel holds a single epilogue
// body: with both in one kernel the compiler moves the accumulators to VGPRs
// ahead of the branch between them and spills.
template <bool kMasked>
struct EpiLse {
  float2* part;   // [vocabulary tile][ldp] (max, sum exp) per token
  int64_t ldp;
  int64_t M;      // valid vocabulary rows of this launch
  int64_t tile0;  // vocabulary tile of this launch's first tile
  TileClock clock;  // measurement hook
  float rm[kNI], rs[kNI];

  __device__ __forceinline__ void mark(int phase) { clock.mark(phase); }

  __device__ __forceinline__ void begin(int64_t, int, int, int) {
#pragma unroll
    for (int i = 0; i < kNI; ++i) {
      rm[i] = -__builtin_inff();
      rs[i] = 0.0f;
    }
  }

  // Running (max, sum exp) per token column over this wave's 128 vocabulary
  // rows; with kMasked, rows at or past the vocabulary end read as -inf. The
  // accumulators themselves are left untouched so they can stay in AGPRs.
  __device__ __forceinline__ void update(const f32x16_t (&acc)[kMI][kNI], int lim) {
    // One token column at a time: its 64 accumulators are read out of their
    // AGPRs into VGPRs, reduced to a max, then to a sum of exponentials.
#pragma unroll
    for (int ni = 0; ni < kNI; ++ni) {
      float z[kMI * 16];
#pragma unroll
      for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int off = mi * 32 + (r & 3) + 8 * (r >> 2);
          const float x = acc_read(acc[mi][ni][r]);
          z[mi * 16 + r] = !kMasked || off < lim ? x : -__builtin_inff();
        }
      float tmax = -__builtin_inff();
#pragma unroll
      for (int i = 0; i < kMI * 16; ++i) tmax = fmaxf(tmax, z[i]);
      const float mn = fmaxf(rm[ni], tmax);
      if (mn != -__builtin_inff()) {
        const float sc = mn * kLog2e;
        float s = rs[ni] * fast_exp2(fmaf(rm[ni], kLog2e, -sc));
#pragma unroll
        for (int i = 0; i < kMI * 16; ++i) s += fast_exp2(fmaf(z[i], kLog2e, -sc));
        rm[ni] = mn;
        rs[ni] = s;
      }
    }
  }

  __device__ __forceinline__ void tile(f32x16_t (&acc)[kMI][kNI], int64_t m0, int64_t, int wm, int,
                                       int lane, void*) {
    if constexpr (kMasked) {
      // Vocabulary rows from this wave's first row; the lane's rows sit at offsets
      // up to 123 past it plus 4 (lane >> 5).
      const int64_t rows = M - m0 - wm * (kBM / 2);
      const int64_t lim64 = rows - 4 * (lane >> 5);
      update(acc, lim64 > kBM ? kBM : static_cast<int>(lim64));
    } else {
      update(acc, kBM);
    }
  }

  __device__ __forceinline__ void finish(int mg, int64_t n0, int wm, int wn, int lane, void* smem) {
    clock.tile_id = ((tile0 + mg) << 32) | (n0 / kBN);
#pragma unroll
    for (int ni = 0; ni < kNI; ++ni) {
      const float m2 = __shfl_xor(rm[ni], 32, 64);
      const float s2 = __shfl_xor(rs[ni], 32, 64);
      lse_merge(rm[ni], rs[ni], m2, s2);
    }
    float2* sh = static_cast<float2*>(smem);
    __syncthreads();
    if (wm == 1 && lane < 32)
#pragma unroll
      for (int ni = 0; ni < kNI; ++ni) sh[acc_col(wn, ni, lane)] = make_float2(rm[ni], rs[ni]);
    __syncthreads();
    if (wm == 0 && lane < 32) {
#pragma unroll
      for (int ni = 0; ni < kNI; ++ni) {
        const float2 o = sh[acc_col(wn, ni, lane)];
        lse_merge(rm[ni], rs[ni], o.x, o.y);
        part[(tile0 + mg) * ldp + n0 + acc_col(wn, ni, lane)] = make_float2(rm[ni], rs[ni]);
      }
    }
  }
};

// With `clk` (a measurement hook, normally null), slot b < clk_slots (by default
// the workgroup, blockIdx.x plus blockIdx.y times gridDim.x) records a tile's
// timeline in clk[8b .. 8b+7]: the hardware ids of its wave 0 (HW_REG_XCC_ID << 32
// | HW_REG_HW_ID), its start and end on the constant wall clock (s_memrealtime),
// the shader clock (s_memtime) at its start, after the prologue, after the K loop
// and at its end, and its tile. c0 and r0 are the start readings.
__device__ __forceinline__ void write_clock_record(int64_t* clk, int64_t clk_slots, uint64_t c0, uint64_t r0,
                                                   const TileClock& tc, int64_t b) {
  if (!clk || threadIdx.x != 0 || b < 0 || b >= clk_slots) return;
  const uint64_t c1 = __builtin_amdgcn_s_memtime();
  const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
  // s_getreg_b32 of the whole HW_ID (register 4) and XCC_ID (register 20)
  const uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);
  const uint32_t xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20);
  int64_t* rec = clk + 8 * b;
  rec[0] = (static_cast<int64_t>(xcc) << 32) | hw;
  rec[1] = static_cast<int64_t>(r0);
  rec[2] = static_cast<int64_t>(r1);
  rec[3] = static_cast<int64_t>(c0);
  rec[4] = static_cast<int64_t>(tc.t_mark[0]);
  rec[5] = static_cast<int64_t>(tc.t_mark[1]);
  rec[6] = static_cast<int64_t>(c1);
  rec[7] = tc.tile_id;
}
__device__ __forceinline__ void write_clock_record(int64_t* clk, int64_t clk_slots, uint64_t c0, uint64_t r0,
                                                   const TileClock& tc) {
  write_clock_record(clk, clk_slots, c0, r0, tc, static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x);
}

// The head forward, with the timeline hook above (the tile is vocabulary tile
// << 32 | token tile).
template <class E, bool kMasked>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_head_fwd(GemmShape s, float2* part, int64_t ldp, int64_t tile0, int64_t* clk, int64_t clk_slots) {
  __shared__ v4u lds[kStages][kStageChunks];
  const uint64_t c0 = clk ? __builtin_amdgcn_s_memtime() : 0;
  const uint64_t r0 = clk ? __builtin_amdgcn_s_memrealtime() : 0;
  EpiLse<kMasked> epi;
  epi.part = part;
  epi.ldp = ldp;
  epi.M = s.m;
  epi.tile0 = tile0;
  epi.clock.start(clk != nullptr);
  gemm_body<E, false, false>(s, epi, lds);
  write_clock_record(clk, clk_slots, c0, r0, epi.clock);
}

// Tile idx (< mx * nv) of an XCD's list in a pulling launch: its vocabulary
// tiles v (v % 8 == xcd, mx of them) against the nv valid token tiles, in groups
// of up to 4 vocabulary tiles, and within a group in waves of up to 8 token tiles,
// vocabulary tile by vocabulary tile. The 32 tiles an XCD runs at once thus share
// 12 operand panels in its L2.
__device__ __forceinline__ void pull_tile(int idx, int mx, int nv, int xcd, int& mt, int& n_tile) {
  const int g = idx / (4 * nv);
  const int msz = mx - 4 * g < 4 ? mx - 4 * g : 4;
  const int rem = idx - g * 4 * nv;
  const int nwave = rem / (msz * 8);
  const int r2 = rem - nwave * msz * 8;
  const int nsz = nv - 8 * nwave < 8 ? nv - 8 * nwave : 8;
  mt = (4 * g + r2 / nsz) * 8 + xcd;
  n_tile = 8 * nwave + r2 % nsz;
}

__global__ __launch_bounds__(256) void k_fill_i64(int64_t* p, int64_t n, int64_t v) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = v;
}

// The head forward as a grid of workgroups (a multiple of 8, normally one per
// CU) that pull tiles until none is left, instead of one workgroup per tile.
// Workgroup b runs on XCD b % 8 and takes, from the XCD's own counter
// next[b % 8] (zeroed before the launch), first the tiles of that XCD's full
// vocabulary tiles (v with v % 8 == b % 8; order of pull_tile), then, when st
// describes a partial last vocabulary tile (st.m > 0), that tile's token tiles
// t with t % 8 == b % 8, with the masked epilogue. Only valid token tiles (below
// the device count) are enumerated, so no workgroup is dispatched for nothing,
// and a workgroup takes its next tile as soon as it is free, whichever shader
// engine it sits on. The timeline hook records tile (v, t) in slot
// v x n_tiles + t (the partial tile as v = s.m_tiles).
template <class E>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_head_fwd_pull(GemmShape s, GemmShape st, float2* part, int64_t ldp, int32_t* next, int64_t* clk,
                     int64_t clk_slots) {
  __shared__ v4u lds[kStages][kStageChunks];
  __shared__ int32_t s_idx;
  const int xcd = static_cast<int>(blockIdx.x & 7);
  const int64_t n_valid = s.n_dev ? static_cast<int64_t>(*s.n_dev) : s.n;
  const int64_t nv64 = (n_valid + kBN - 1) / kBN;
  const int nv = static_cast<int>(nv64 < s.n_tiles ? nv64 : s.n_tiles);        // valid token tiles
  const int mx = xcd < s.m_tiles ? (s.m_tiles - 1 - xcd) / 8 + 1 : 0;            // this XCD's vocabulary tiles
  const int32_t total = mx * nv;
  // then the partial last vocabulary tile's token tiles t with t % 8 == xcd (st.m > 0)
  const int32_t tail = st.m > 0 && xcd < nv ? (nv - 1 - xcd) / 8 + 1 : 0;
  EpiLse<false> epi;
  epi.part = part;
  epi.ldp = ldp;
  epi.M = s.m;
  epi.tile0 = 0;
  EpiLse<true> epi_t;
  epi_t.part = part;
  epi_t.ldp = ldp;
  epi_t.M = st.m;
  epi_t.tile0 = s.m_tiles;
  for (;;) {
    if (threadIdx.x == 0) s_idx = atomicAdd(next + xcd, 1);
    __syncthreads();  // also: the previous tile's epilogue is done with LDS
    const int32_t idx = s_idx;
    __syncthreads();  // every thread has read s_idx
    if (idx >= total + tail) break;
    if (idx >= total) {
      const int n_tile = (idx - total) * 8 + xcd;
      const uint64_t c0 = clk ? __builtin_amdgcn_s_memtime() : 0;
      const uint64_t r0 = clk ? __builtin_amdgcn_s_memrealtime() : 0;
      epi_t.clock.start(clk != nullptr);
      gemm_tile<E, false, false>(st, epi_t, lds, 0, n_tile);
      write_clock_record(clk, clk_slots, c0, r0, epi_t.clock, static_cast<int64_t>(s.m_tiles) * s.n_tiles + n_tile);
      continue;
    }
    int mt, n_tile;
    pull_tile(idx, mx, nv, xcd, mt, n_tile);
    const uint64_t c0 = clk ? __builtin_amdgcn_s_memtime() : 0;
    const uint64_t r0 = clk ? __builtin_amdgcn_s_memrealtime() : 0;
    epi.clock.start(clk != nullptr);
    gemm_tile<E, false, false>(s, epi, lds, mt, n_tile);
    write_clock_record(clk, clk_slots, c0, r0, epi.clock, static_cast<int64_t>(mt) * s.n_tiles + n_tile);
  }
}

template <class E>
__device__ __forceinline__ float dot_chunk(const v4u& a, const v4u& b);

template <>
__device__ __forceinline__ float dot_chunk<BF16>(const v4u& a, const v4u& b) {
  const uint32_t* x = reinterpret_cast<const uint32_t*>(&a);
  const uint32_t* y = reinterpret_cast<const uint32_t*>(&b);
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    s = fmaf(__uint_as_float(x[i] << 16), __uint_as_float(y[i] << 16), s);
    s = fmaf(__uint_as_float(x[i] & 0xffff0000u), __uint_as_float(y[i] & 0xffff0000u), s);
  }
  return s;
}

template <>
__device__ __forceinline__ float dot_chunk<F32>(const v4u& a, const v4u& b) {
  float s = __uint_as_float(a.x) * __uint_as_float(b.x);
  s = fmaf(__uint_as_float(a.y), __uint_as_float(b.y), s);
  s = fmaf(__uint_as_float(a.z), __uint_as_float(b.z), s);
  s = fmaf(__uint_as_float(a.w), __uint_as_float(b.w), s);
  return s;
}

// 64 compacted rows per block, lane l of every wave on row l. Phase 1: wave w
// merges the row's partials of vocabulary tiles w, w + 4, w + 8, ... in that
// order (8 loads in flight; the 64 lanes read 256 contiguous bytes of a tile's
// partials, [tile][row]), then the four waves' results are merged in wave order.
// Phase 2: the target logits as dot products, 8 lanes per row and 8 rows per
// wave at a time (each lane takes every 8th 16-byte chunk of the row), then
// logp = z_y - lse at the row's position.
constexpr int kFinRows = 64;
template <class E>
__global__ __launch_bounds__(256) void k_fwd_finalize(const float2* part, int64_t ldp, int m_groups,
                                                      const typename E::storage* hc, int64_t H,
                                                      const typename E::storage* w, int64_t ld_w,
                                                      int64_t V, const int32_t* idx,
                                                      const int32_t* target, const int32_t* count,
                                                      float* logp, float* lse, int32_t* status) {
  constexpr int kWaves = 4;
  constexpr int kInFlight = 8;
  __shared__ float2 s_ms[kWaves][kFinRows];
  __shared__ float s_lse[kFinRows];
  const int64_t n = *count;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kFinRows;
  if (c0 >= n) return;  // uniform over the block
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  {
    const int64_t c = c0 + lane;
    float m = -__builtin_inff(), s = 0.0f;
    if (c < n) {
      int gi = wave;
      for (; gi + (kInFlight - 1) * kWaves < m_groups; gi += kInFlight * kWaves) {
        float2 p[kInFlight];
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) p[u] = part[static_cast<int64_t>(gi + u * kWaves) * ldp + c];
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) lse_merge(m, s, p[u].x, p[u].y);
      }
      for (; gi < m_groups; gi += kWaves) {
        const float2 p = part[static_cast<int64_t>(gi) * ldp + c];
        lse_merge(m, s, p.x, p.y);
      }
    }
    s_ms[wave][lane] = make_float2(m, s);
  }
  __syncthreads();
  if (wave == 0) {
    float m = s_ms[0][lane].x, s = s_ms[0][lane].y;
#pragma unroll
    for (int q = 1; q < kWaves; ++q) lse_merge(m, s, s_ms[q][lane].x, s_ms[q][lane].y);
    s_lse[lane] = m + logf(s);
  }
  __syncthreads();
  const int sub = lane & 7;                 // lane within the row's group of 8
  const int64_t chunks = H / E::kPerChunk;  // 16-byte chunks per row
  for (int j = 0; j < kFinRows / kWaves; j += 8) {
    const int r = wave * (kFinRows / kWaves) + j + (lane >> 3);  // row of this block
    const int64_t c = c0 + r;
    float z = 0.0f;
    int64_t t = 0;
    bool yok = false;
    if (c < n) {
      t = idx[c];
      const int32_t y = target[t];
      yok = y >= 0 && static_cast<int64_t>(y) < V;
      if (yok) {
        const v4u* hr = reinterpret_cast<const v4u*>(hc + c * H);
        const v4u* wr = reinterpret_cast<const v4u*>(w + static_cast<int64_t>(y) * ld_w);
        for (int64_t k = sub; k < chunks; k += 8) z += dot_chunk<E>(hr[k], wr[k]);
      }
    }
    z += __shfl_xor(z, 4, 64);
    z += __shfl_xor(z, 2, 64);
    z += __shfl_xor(z, 1, 64);
    if (sub == 0 && c < n) {
      const float l = s_lse[r];
      const bool finite = __builtin_isfinite(l);
      if (status && !yok) atomicOr(status, SAO_STATUS_TARGET_RANGE);
      if (status && !finite) atomicOr(status, SAO_STATUS_NONFINITE);
      lse[t] = l;
      logp[t] = yok ? z - l : __builtin_nanf("");
    }
  }
}

// ------------------------------------------------------------------------- //
// Backward
// ------------------------------------------------------------------------- //
template <class E>
__device__ __forceinline__ void store4(typename E::storage* p, const float (&d)[4]);

template <>
__device__ __forceinline__ void store4<BF16>(uint16_t* p, const float (&d)[4]) {
  const uint32_t lo = pack_bf16x2(d[0], d[1]);
  const uint32_t hi = pack_bf16x2(d[2], d[3]);
  *reinterpret_cast<uint2*>(p) = make_uint2(lo, hi);
}

template <>
__device__ __forceinline__ void store4<F32>(float* p, const float (&d)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(d[0], d[1], d[2], d[3]);
}


// dz_{t,v} = g_t (1[v = y_t] - exp(z_{t,v} - lse_t)) for one vocabulary block, stored
// token-major dz[c][v - v0] (row stride ldz). The dH product reads it K-major, the
// dW product MN-major, so no transposed copy is written. Columns past the block's
// valid vocabulary rows hold zeros. kMasked: the launch covers the block's last,
// partial vocabulary tile (a launch of its own, like the forward's).
template <class E, bool kMasked>
struct EpiDz {
  typename E::storage* dz;
  int64_t ldz;
  int64_t m_valid;   // vocabulary rows of this block
  int64_t v_base;    // vocabulary index of block row 0
  const float* g_c;
  const float* lse_c;
  const int32_t* y_c;
  float gl[kNI], ll[kNI];
  int64_t yl[kNI];
  int yt[kNI];  // target row of the column's token inside the current tile, or -8 when outside
  TileClock clock;  // measurement hook

  __device__ __forceinline__ void mark(int phase) { clock.mark(phase); }

  __device__ __forceinline__ void begin(int64_t n0, int, int wn, int lane) {
#pragma unroll
    for (int ni = 0; ni < kNI; ++ni) {
      const int64_t c = n0 + acc_col(wn, ni, lane);
      gl[ni] = g_c[c];
      ll[ni] = lse_c[c] * kLog2e;
      yl[ni] = static_cast<int64_t>(y_c[c]) - v_base;
    }
  }

  // dz of accumulator (mi, ni, registers 4j .. 4j+3): four consecutive
  // vocabulary rows starting at tile row vt. dz = g (onehot - p): the target
  // row of a token lies in a given tile rarely, so the one-hot term is a branch
  // on yt (the target's tile row, or far outside), and rows at or past the end
  // of the block (last tile only, kMasked) are zero.
  __device__ __forceinline__ void dz4(const f32x16_t (&acc)[kMI][kNI], int mi, int ni, int j, int vt,
                                      int rows, float (&d)[4]) const {
    float p[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      p[e] = fast_exp2(fmaf(acc_read(acc[mi][ni][4 * j + e]), kLog2e, -ll[ni]));
      d[e] = gl[ni] * -p[e];
    }
    const unsigned k = static_cast<unsigned>(yt[ni] - vt);
    if (k < 4u) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (static_cast<unsigned>(e) == k) d[e] = gl[ni] * (1.0f - p[e]);
    }
    if constexpr (kMasked) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (vt + e >= rows) d[e] = 0.0f;
    }
  }

  __device__ __forceinline__ void tile(f32x16_t (&acc)[kMI][kNI], int64_t m0, int64_t n0, int wm, int wn,
                                       int lane, void*) {
    clock.tile_id = ((m0 / kBM) << 32) | (n0 / kBN);
    // Valid rows of this tile (all 256 unless kMasked).
    const int64_t rows64 = m_valid - m0;
    const int rows = rows64 > kBM ? kBM : static_cast<int>(rows64);
#pragma unroll
    for (int ni = 0; ni < kNI; ++ni) {
      const int64_t y = yl[ni] - m0;
      yt[ni] = y >= 0 && y < kBM ? static_cast<int>(y) : -8;
    }
    if constexpr (sizeof(typename E::storage) == 2) {
      // Straight from the accumulators with 16-byte stores. Of the register
      // groups j = 2p and 2p + 1 (vocabulary rows 16p + 4h .. +3 and 16p + 8 + 4h
      // .. +3 of lane half h), v_permlane32_swap trades group 2p of the upper
      // half for group 2p + 1 of the lower half, so that each lane holds 8
      // consecutive rows (16p + 8h ..) of its token: one 16-byte chunk.
#pragma unroll
      for (int ni = 0; ni < kNI; ++ni) {
        typename E::storage* row = dz + (n0 + acc_col(wn, ni, lane)) * ldz + m0;
#pragma unroll
        for (int mi = 0; mi < kMI; ++mi) {
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            float d0[4], d1[4];
            dz4(acc, mi, ni, 2 * p, acc_row(wm, mi, 8 * p, lane), rows, d0);
            dz4(acc, mi, ni, 2 * p + 1, acc_row(wm, mi, 8 * p + 4, lane), rows, d1);
            const auto lo = __builtin_amdgcn_permlane32_swap(pack_bf16x2(d0[0], d0[1]), pack_bf16x2(d1[0], d1[1]),
                                                             false, false);
            const auto hi = __builtin_amdgcn_permlane32_swap(pack_bf16x2(d0[2], d0[3]), pack_bf16x2(d1[2], d1[3]),
                                                             false, false);
            const int v = wm * (kBM / 2) + mi * 32 + 16 * p + 8 * (lane >> 5);
            *reinterpret_cast<v4u*>(row + v) = v4u{lo[0], hi[0], lo[1], hi[1]};
          }
        }
      }
    } else {
#pragma unroll
      for (int ni = 0; ni < kNI; ++ni) {
        const int64_t c = n0 + acc_col(wn, ni, lane);
        typename E::storage* row = dz + c * ldz;
#pragma unroll
        for (int mi = 0; mi < kMI; ++mi) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int vl = acc_row(wm, mi, 4 * j, lane);
            float d[4];
            dz4(acc, mi, ni, j, vl, rows, d);
            store4<E>(row + m0 + vl, d);
          }
        }
      }
    }
  }

  __device__ __forceinline__ void finish(int, int64_t, int, int, int, void*) {}
};

// out[m][n] += acc (fp32), rows < m_valid and columns < n_valid. Each element has
// one writer per launch and launches on a stream are ordered, so a plain load,
// add and store per element is an exact, deterministic accumulate. The loads of
// one 32-column block (64 per lane) are issued together, so that a tile pays a
// few load latencies instead of a stream of read-modify-write atomics in L2
// (every tile of a round reaches its epilogue at about the same time).
struct EpiAcc {
  float* out;
  int64_t ldo;
  int64_t m_valid;
  int64_t n_valid;
  int64_t split_stride;  // elements between the outputs of successive K pieces
  bool overwrite;        // store the tile instead of adding it (the first contribution)
  TileClock clock;       // measurement hook

  __device__ __forceinline__ void mark(int phase) { clock.mark(phase); }

  __device__ __forceinline__ void begin(int64_t, int, int, int) {}

  __device__ __forceinline__ void tile(f32x16_t (&acc)[kMI][kNI], int64_t m0, int64_t n0, int wm, int wn,
                                       int lane, void*) {
    clock.tile_id = ((m0 / kBM) << 32) | (n0 / kBN);
    const bool whole = m0 + kBM <= m_valid && n0 + kBN <= n_valid;  // uniform
    if (whole) {
      // Element (mi, ni, r) sits at a uniform base (the wave's 32-row block of
      // mi and its 32 columns of ni) plus a uniform row offset of r plus this
      // lane's fixed offset, so the loads and stores take a scalar base and one
      // address register (global address space, so that they are not flat).
      using gchar = __attribute__((address_space(1))) char;
      const uint32_t lane_off = static_cast<uint32_t>((4 * (lane >> 5) * ldo + (lane & 31)) * 4);
      if (overwrite) {
#pragma unroll
        for (int ni = 0; ni < kNI; ++ni)
#pragma unroll
          for (int mi = 0; mi < kMI; ++mi) {
            gchar* b = (gchar*)uniform_ptr(out + (m0 + wm * (kBM / 2) + mi * 32) * ldo + n0 +
                                           wn * (kBN / kWavesN) + ni * 32);
#pragma unroll
            for (int r = 0; r < 16; ++r)
              *(__attribute__((address_space(1))) float*)(b + ((r & 3) + 8 * (r >> 2)) * ldo * 4 + lane_off) =
                  acc_read(acc[mi][ni][r]);
          }
        return;
      }
#pragma unroll
      for (int ni = 0; ni < kNI; ++ni) {
        float v[kMI][16];
#pragma unroll
        for (int mi = 0; mi < kMI; ++mi) {
          gchar* b = (gchar*)uniform_ptr(out + (m0 + wm * (kBM / 2) + mi * 32) * ldo + n0 + wn * (kBN / kWavesN) +
                                         ni * 32);
#pragma unroll
          for (int r = 0; r < 16; ++r)
            v[mi][r] = *(__attribute__((address_space(1))) const float*)(b + ((r & 3) + 8 * (r >> 2)) * ldo * 4 +
                                                                         lane_off);
        }
#pragma unroll
        for (int mi = 0; mi < kMI; ++mi) {
          gchar* b = (gchar*)uniform_ptr(out + (m0 + wm * (kBM / 2) + mi * 32) * ldo + n0 + wn * (kBN / kWavesN) +
                                         ni * 32);
#pragma unroll
          for (int r = 0; r < 16; ++r)
            *(__attribute__((address_space(1))) float*)(b + ((r & 3) + 8 * (r >> 2)) * ldo * 4 + lane_off) =
                v[mi][r] + acc_read(acc[mi][ni][r]);
        }
      }
      return;
    }
#pragma unroll
    for (int ni = 0; ni < kNI; ++ni) {
      const int64_t n = n0 + acc_col(wn, ni, lane);
      if (n >= n_valid) continue;
#pragma unroll
      for (int mi = 0; mi < kMI; ++mi)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t m = m0 + acc_row(wm, mi, r, lane);
          if (m < m_valid) out[m * ldo + n] = acc_read(acc[mi][ni][r]) + (overwrite ? 0.0f : out[m * ldo + n]);
        }
    }
  }

  __device__ __forceinline__ void finish(int, int64_t, int, int, int, void*) {}
};

template <class E, bool kMasked>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_bwd_dz(GemmShape s, EpiDz<E, kMasked> epi, int64_t* clk, int64_t clk_slots) {
  __shared__ v4u lds[kStages][kStageChunks];
  const uint64_t c0 = clk ? __builtin_amdgcn_s_memtime() : 0;
  const uint64_t r0 = clk ? __builtin_amdgcn_s_memrealtime() : 0;
  epi.clock.start(clk != nullptr);
  gemm_body<E, false, false>(s, epi, lds);
  write_clock_record(clk, clk_slots, c0, r0, epi.clock);
}

// The logit recompute of one vocabulary block as a pulling launch (at up to 8192
// tokens), with the block's partial last tile (st.m > 0) taken after each XCD's
// full tiles: the same tile lists as the pulling head forward. Tile (v, t) of the
// block records in slot v x n_tiles + t.
template <class E>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_bwd_dz_pull(GemmShape s, GemmShape st, EpiDz<E, false> epi, EpiDz<E, true> epi_t, int32_t* next,
                   int64_t* clk, int64_t clk_slots) {
  __shared__ v4u lds[kStages][kStageChunks];
  __shared__ int32_t s_idx;
  const int xcd = static_cast<int>(blockIdx.x & 7);
  const int64_t n_valid = s.n_dev ? static_cast<int64_t>(*s.n_dev) : s.n;
  const int64_t nv64 = (n_valid + kBN - 1) / kBN;
  const int nv = static_cast<int>(nv64 < s.n_tiles ? nv64 : s.n_tiles);
  const int mx = xcd < s.m_tiles ? (s.m_tiles - 1 - xcd) / 8 + 1 : 0;
  const int32_t total = mx * nv;
  const int32_t tail = st.m > 0 && xcd < nv ? (nv - 1 - xcd) / 8 + 1 : 0;
  for (;;) {
    if (threadIdx.x == 0) s_idx = atomicAdd(next + xcd, 1);
    __syncthreads();  // also: the previous tile's epilogue is done with LDS
    const int32_t idx = s_idx;
    __syncthreads();  // every thread has read s_idx
    if (idx >= total + tail) break;
    const uint64_t c0 = clk ? __builtin_amdgcn_s_memtime() : 0;
    const uint64_t r0 = clk ? __builtin_amdgcn_s_memrealtime() : 0;
    if (idx >= total) {
      const int n_tile = (idx - total) * 8 + xcd;
      epi_t.clock.start(clk != nullptr);
      gemm_tile<E, false, false>(st, epi_t, lds, 0, n_tile);
      // the record names the tile within the block, not within the tail's own shape
      if (epi_t.clock.tile_id >= 0) epi_t.clock.tile_id += static_cast<int64_t>(s.m_tiles) << 32;
      write_clock_record(clk, clk_slots, c0, r0, epi_t.clock, static_cast<int64_t>(s.m_tiles) * s.n_tiles + n_tile);
      continue;
    }
    int mt, n_tile;
    pull_tile(idx, mx, nv, xcd, mt, n_tile);
    epi.clock.start(clk != nullptr);
    gemm_tile<E, false, false>(s, epi, lds, mt, n_tile);
    write_clock_record(clk, clk_slots, c0, r0, epi.clock, static_cast<int64_t>(mt) * s.n_tiles + n_tile);
  }
}

// dH += dz . W (dz K-major, W MN-major) and dW += dz^T . Hg (both MN-major).
template <class E, bool AMn, bool BMn>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_bwd_acc(GemmShape s, EpiAcc epi, int64_t* clk, int64_t clk_slots) {
  __shared__ v4u lds[kStages][kStageChunks];
  const uint64_t c0 = clk ? __builtin_amdgcn_s_memtime() : 0;
  const uint64_t r0 = clk ? __builtin_amdgcn_s_memrealtime() : 0;
  epi.clock.start(clk != nullptr);
  epi.out += static_cast<int64_t>(blockIdx.y) * epi.split_stride;  // this K piece's own output
  gemm_body<E, AMn, BMn>(s, epi, lds);
  write_clock_record(clk, clk_slots, c0, r0, epi.clock);
}


// Zero rows [0, round_up(count, kRowPad)) of accumulators q0 .. pieces - 1, `stride`
// floats apart.
__global__ __launch_bounds__(256) void k_zero_rows(float* p, int64_t H, const int32_t* count, int q0, int pieces,
                                                   int64_t stride) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (c >= round_up_dev(*count, kRowPad)) return;
  for (int q = q0; q < pieces; ++q) {
    float4* r = reinterpret_cast<float4*>(p + q * stride + c * H);
    for (int64_t k = threadIdx.x & 63; k < H / 4; k += 64) r[k] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

// dhidden[t] = sum over the K pieces (in order) of dH[pos[t]], rounded to the
// element type, or zeros when pos[t] < 0.
template <class E>
__global__ __launch_bounds__(256) void k_dh_scatter(const float* dh, int64_t H, const int32_t* pos,
                                                    int64_t T, int pieces, int64_t stride,
                                                    typename E::storage* dhid) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int32_t c = pos[t];
  typename E::storage* out = dhid + t * H;
  for (int64_t k = threadIdx.x & 63; k < H / 4; k += 64) {
    float d[4] = {0.f, 0.f, 0.f, 0.f};
    if (c >= 0) {
      for (int q = 0; q < pieces; ++q) {
        const float4 v = reinterpret_cast<const float4*>(dh + q * stride + static_cast<int64_t>(c) * H)[k];
        d[0] += v.x; d[1] += v.y; d[2] += v.z; d[3] += v.w;
      }
    }
    store4<E>(out + 4 * k, d);
  }
}

// ------------------------------------------------------------------------- //
// Launchers
// ------------------------------------------------------------------------- //
static GemmShape make_shape(const void* a, int64_t lda, int64_t m, const void* b, int64_t ldb, int64_t n,
                            int64_t k) {
  GemmShape s{};
  s.a = a; s.lda = lda; s.m = m;
  s.b = b; s.ldb = ldb; s.n = n;
  s.k = k;
  s.m_tiles = static_cast<int>(ceil_div(m, kBM));
  s.n_tiles = static_cast<int>(ceil_div(n, kBN));
  // Few N tiles (a token chunk against the whole vocabulary): split M across the
  // XCDs, so each XCD streams its own share of A while the small B is shared.
  // Otherwise split N, so that the 8 XCDs read each A panel together.
  s.msplit = s.n_tiles <= kMsplitMaxNTiles ? 1 : 0;
  s.sn = s.msplit ? pick_sn_msplit(s.n_tiles) : pick_sn(s.n_tiles);
  return s;
}

// Host-bound token tiles up to which the forward and the backward's logit
// recompute pull their tiles (k_head_fwd_pull, k_bwd_dz_pull) rather than
// launching one workgroup per tile of the host bound. Measured per workload
// against the one-workgroup-per-tile raster: on an 8192-token chunk (32
// host-bound tiles, about 16 with loss-mask rows) the forward 7 % faster and
// the recompute 6 %; the forward at 32,768 tokens and H = 6144 (128 tiles) 4 %
// slower, at 65,536 tokens (256) 0.7 % slower.
constexpr int kPullMaxNTiles = 32;

// Workgroups of a pulling launch: one per CU of the current device, rounded
// down to a multiple of 8 (the XCDs), at least 8.
static int pull_grid() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 256;
  cus = cus / 8 * 8;
  return cus < 8 ? 8 : cus;
}

template <class E>
static hipError_t logprob_impl(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w,
                               const int32_t* target, const uint8_t* mask, int64_t T, int64_t H,
                               int64_t V, float* logp, float* lse, int32_t* status, void* ws,
                               hipStream_t st) {
  using S = typename E::storage;
  const LogprobLayout L = logprob_layout(T, H, V, sizeof(S));
  char* w8 = static_cast<char*>(ws);
  int32_t* blk = reinterpret_cast<int32_t*>(w8 + L.blk_counts);
  int32_t* count = reinterpret_cast<int32_t*>(w8 + L.count);
  int32_t* idx = reinterpret_cast<int32_t*>(w8 + L.idx);
  S* hc = reinterpret_cast<S*>(w8 + L.hc);
  float2* part = reinterpret_cast<float2*>(w8 + L.part);

  const int nb = static_cast<int>(L.n_count_blocks);
  int32_t* next = reinterpret_cast<int32_t*>(w8 + L.next);
  hipLaunchKernelGGL(k_count_rows, dim3(nb), dim3(256), 0, st, mask, nullptr, T, blk, next, 8);
  hipLaunchKernelGGL(k_compact_rows, dim3(nb), dim3(256), 0, st, mask, nullptr, T, blk, idx,
                     nullptr, count, logp, lse);
  const int rows4 = static_cast<int>(L.t_pad / 4);
  hipLaunchKernelGGL(k_gather_rows<E>, dim3(rows4), dim3(256), 0, st, static_cast<const S*>(hidden),
                     ld_hidden, H, idx, count, hc, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
  // The vocabulary tiles with 256 valid rows, then (when V is not a multiple of
  // 256) the last, partial tile in a launch of its own with the masked epilogue.
  const int64_t full_tiles = V / kBM;
  const int64_t rem = V - full_tiles * kBM;
  const KernelTimer& tm = kernel_timer();
  const bool timed = tm.timed(SAO_KERNEL_HEAD_FORWARD);
  if (timed) (void)hipEventRecord(tm.start, st);
  // The forward splits the vocabulary across the XCDs (M-split) whatever the
  // token count: each XCD streams its own W panels while all of them read the
  // same hidden rows, which the memory-side cache holds (measured 0.7 % faster
  // than splitting the tokens at 65,536 tokens).
  bool tail_done = false;
  if (full_tiles > 0) {
    GemmShape s = make_shape(w_head, ld_w, full_tiles * kBM, hc, H, T, H);
    s.n_dev = count;
    int64_t* clk = tm.clocks_for(SAO_KERNEL_HEAD_FORWARD);
    if (s.n_tiles <= kPullMaxNTiles) {
      // The pulling kernel records by tile, not by workgroup: clear the records
      // first, so that this launch's are the only ones left.
      if (clk)
        hipLaunchKernelGGL(k_fill_i64, dim3(64), dim3(256), 0, st, clk, 8 * tm.clock_slots, int64_t{0});
      // It also takes the partial last vocabulary tile's tiles, at the end of each XCD's list.
      GemmShape stail{};
      if (rem > 0) {
        stail = make_shape(static_cast<const S*>(w_head) + full_tiles * kBM * ld_w, ld_w, rem, hc, H, T, H);
        stail.n_dev = count;
      }
      hipLaunchKernelGGL(k_head_fwd_pull<E>, dim3(static_cast<unsigned>(pull_grid())), dim3(kThreads), 0, st, s,
                         stail, part, L.t_pad, next, clk, tm.clock_slots);
      tail_done = true;
    } else {
      s.msplit = 1;
      s.sn = pick_sn_msplit(s.n_tiles);
      hipLaunchKernelGGL((k_head_fwd<E, false>), dim3(gemm_grid(s)), dim3(kThreads), 0, st, s, part, L.t_pad,
                         int64_t{0}, clk, tm.clock_slots);
    }
  }
  if (rem > 0 && !tail_done) {
    // A single row of tiles: the M-split raster would deal its one M tile to one
    // XCD, so the tiles are dealt out along N (make_shape's choice for many token
    // tiles) and spread over all 8 XCDs.
    GemmShape s = make_shape(static_cast<const S*>(w_head) + full_tiles * kBM * ld_w, ld_w, rem, hc, H, T, H);
    s.n_dev = count;
    hipLaunchKernelGGL((k_head_fwd<E, true>), dim3(gemm_grid(s)), dim3(kThreads), 0, st, s, part, L.t_pad,
                       full_tiles, static_cast<int64_t*>(nullptr), int64_t{0});
  }
  if (timed) (void)hipEventRecord(tm.stop, st);
  hipLaunchKernelGGL(k_fwd_finalize<E>, dim3(static_cast<unsigned>(L.t_pad / kFinRows)), dim3(256), 0, st, part,
                     L.t_pad,
                     static_cast<int>(L.m_tiles), hc, H, static_cast<const S*>(w_head), ld_w, V, idx,
                     target, count, logp, lse, status);
  return hipGetLastError();
}

template <class E>
static hipError_t backward_impl(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w,
                                const int32_t* target, const float* lse, const float* g, int64_t T,
                                int64_t H, int64_t V, void* dhidden, float* dw, void* ws,
                                hipStream_t st) {
  using S = typename E::storage;
  const BackwardLayout L = backward_layout(T, H, V, sizeof(S));
  char* w8 = static_cast<char*>(ws);
  int32_t* blk = reinterpret_cast<int32_t*>(w8 + L.blk_counts);
  int32_t* count = reinterpret_cast<int32_t*>(w8 + L.count);
  int32_t* idx = reinterpret_cast<int32_t*>(w8 + L.idx);
  int32_t* pos = reinterpret_cast<int32_t*>(w8 + L.pos);
  float* g_c = reinterpret_cast<float*>(w8 + L.g_c);
  float* lse_c = reinterpret_cast<float*>(w8 + L.lse_c);
  int32_t* y_c = reinterpret_cast<int32_t*>(w8 + L.y_c);
  S* hg = reinterpret_cast<S*>(w8 + L.hg);
  float* dh = reinterpret_cast<float*>(w8 + L.dh);
  S* dz = reinterpret_cast<S*>(w8 + L.dz);
  const S* w = static_cast<const S*>(w_head);

  const int nb = static_cast<int>(L.n_count_blocks);
  int32_t* next = reinterpret_cast<int32_t*>(w8 + L.next);  // 8 tile counters per vocabulary block
  hipLaunchKernelGGL(k_count_rows, dim3(nb), dim3(256), 0, st, nullptr, g, T, blk, next,
                     static_cast<int>(8 * L.n_vblocks));
  hipLaunchKernelGGL(k_compact_rows, dim3(nb), dim3(256), 0, st, nullptr, g, T, blk, idx, pos, count,
                     nullptr, nullptr);
  const int rows4 = static_cast<int>(L.t_pad / 4);
  hipLaunchKernelGGL(k_gather_rows<E>, dim3(rows4), dim3(256), 0, st, static_cast<const S*>(hidden),
                     ld_hidden, H, idx, count, hg, target, y_c, g, g_c, lse, lse_c);
  const int64_t dh_stride = L.t_pad * H;
  // dH's K pieces for a block of vlen rows (each piece has its own accumulator).
  auto dh_split = [&](int64_t vlen) { return L.dh_pieces > 1 ? round_up(ceil_div(vlen, L.dh_pieces), 64) : int64_t{0}; };
  auto dh_pieces_of = [&](int64_t vlen) {
    return L.dh_pieces > 1 ? static_cast<int>(ceil_div(vlen, dh_split(vlen))) : 1;
  };
  // The first vocabulary block stores its dH tiles rather than adding them, so
  // only accumulators it has no K piece for need zeros. (Rows past the count in
  // the last token tile are written too, with values nothing reads.)
  const int first_pieces = dh_pieces_of(V < L.vc ? V : L.vc);
  if (first_pieces < L.dh_pieces)
    hipLaunchKernelGGL(k_zero_rows, dim3(rows4), dim3(256), 0, st, dh, H, count, first_pieces, L.dh_pieces,
                       dh_stride);

  // The measurement hooks apply to the first vocabulary block's launches.
  const KernelTimer& tm = kernel_timer();
  auto hook = [&](int64_t vb, int kernel, bool stop_event) {
    if (vb == 0 && tm.timed(kernel)) (void)hipEventRecord(stop_event ? tm.stop : tm.start, st);
  };
  auto clocks = [&](int64_t vb, int kernel) { return vb == 0 ? tm.clocks_for(kernel) : nullptr; };
  for (int64_t vb = 0; vb < L.n_vblocks; ++vb) {
    const int64_t v0 = vb * L.vc;
    const int64_t vlen = (V - v0) < L.vc ? (V - v0) : L.vc;
    // (A) z^T[v][t] = W[v0 + v] . Hg[t] -> dz[t][v]: the block's tiles with 256 valid
    // vocabulary rows, then its partial last tile (if any) with the masked epilogue.
    const int64_t full_v = vlen / kBM * kBM;
    bool tail_done = false;
    if (full_v > 0) {
      GemmShape sa = make_shape(w + v0 * ld_w, ld_w, full_v, hg, H, T, H);
      sa.n_dev = count;
      // A block of W larger than the memory-side cache is streamed once per XCD
      // (M-split) rather than read by all XCDs together (measured at H = 6144:
      // 1.5 ms faster per step; at H = 2048, where the block fits, 0.7 ms slower).
      if (full_v * H * static_cast<int64_t>(sizeof(S)) > kMemorySideCacheBytes) {
        sa.msplit = 1;
        sa.sn = pick_sn_msplit(sa.n_tiles);
      }
      EpiDz<E, false> ez{dz, L.vc, full_v, v0, g_c, lse_c, y_c, {}, {}, {}, {}, {}};
      int64_t* clk = clocks(vb, SAO_KERNEL_BACKWARD_DZ);
      hook(vb, SAO_KERNEL_BACKWARD_DZ, false);
      if (sa.n_tiles <= kPullMaxNTiles) {
        // Few token tiles: tiles pulled per XCD, as in the head forward, the
        // block's partial last tile included.
        GemmShape stail{};
        EpiDz<E, true> ezt{};
        if (vlen > full_v) {
          stail = make_shape(w + (v0 + full_v) * ld_w, ld_w, vlen - full_v, hg, H, T, H);
          stail.n_dev = count;
          ezt = EpiDz<E, true>{dz + full_v, L.vc, vlen - full_v, v0 + full_v, g_c, lse_c, y_c, {}, {}, {}, {}, {}};
        }
        if (clk) hipLaunchKernelGGL(k_fill_i64, dim3(64), dim3(256), 0, st, clk, 8 * tm.clock_slots, int64_t{0});
        hipLaunchKernelGGL(k_bwd_dz_pull<E>, dim3(static_cast<unsigned>(pull_grid())), dim3(kThreads), 0, st, sa,
                           stail, ez, ezt, next + 8 * vb, clk, tm.clock_slots);
        tail_done = true;
      } else {
        hipLaunchKernelGGL((k_bwd_dz<E, false>), dim3(gemm_grid(sa)), dim3(kThreads), 0, st, sa, ez, clk,
                           tm.clock_slots);
      }
      hook(vb, SAO_KERNEL_BACKWARD_DZ, true);
    }
    if (vlen > full_v && !tail_done) {
      GemmShape sa = make_shape(w + (v0 + full_v) * ld_w, ld_w, vlen - full_v, hg, H, T, H);
      sa.n_dev = count;
      EpiDz<E, true> ez{dz + full_v, L.vc, vlen - full_v, v0 + full_v, g_c, lse_c, y_c, {}, {}, {}, {}, {}};
      hipLaunchKernelGGL((k_bwd_dz<E, true>), dim3(gemm_grid(sa)), dim3(kThreads), 0, st, sa, ez,
                         static_cast<int64_t*>(nullptr), int64_t{0});
    }
    // (B) dH[t][h] += sum_v dz[t][v] W[v0 + v][h]: A = dz K-major, B = W MN-major
    // With few token rows the dH tiles cannot fill the GPU: K (the vocabulary)
    // is cut into dh_pieces pieces, each adding into its own accumulator.
    GemmShape sb = make_shape(dz, L.vc, T, w + v0 * ld_w, ld_w, H, vlen);
    sb.m_dev = count;
    sb.msplit = 1;
    sb.sn = pick_sn_msplit(sb.n_tiles);
    sb.k_split = dh_split(vlen);
    const int pieces_b = dh_pieces_of(vlen);
    EpiAcc eb{dh, H, L.t_pad, H, dh_stride, vb == 0, {}};
    hook(vb, SAO_KERNEL_BACKWARD_DH, false);
    hipLaunchKernelGGL((k_bwd_acc<E, false, true>), dim3(gemm_grid(sb), pieces_b), dim3(kThreads), 0, st, sb,
                       eb, clocks(vb, SAO_KERNEL_BACKWARD_DH), tm.clock_slots);
    hook(vb, SAO_KERNEL_BACKWARD_DH, true);
    // (C) dW[v0 + v][h] += sum_t dz[t][v] Hg[t][h]: both MN-major
    GemmShape sc = make_shape(dz, L.vc, vlen, hg, H, H, T);
    sc.k_dev = count;
    sc.msplit = 1;
    sc.sn = pick_sn_msplit(sc.n_tiles);
    EpiAcc ec{dw + v0 * H, H, vlen, H, 0, false, {}};
    hook(vb, SAO_KERNEL_BACKWARD_DW, false);
    hipLaunchKernelGGL((k_bwd_acc<E, true, true>), dim3(gemm_grid(sc)), dim3(kThreads), 0, st, sc, ec,
                       clocks(vb, SAO_KERNEL_BACKWARD_DW), tm.clock_slots);
    hook(vb, SAO_KERNEL_BACKWARD_DW, true);
  }
  const int t4 = static_cast<int>(ceil_div(T, 4));
  hipLaunchKernelGGL(k_dh_scatter<E>, dim3(t4), dim3(256), 0, st, dh, H, pos, T, L.dh_pieces, dh_stride,
                     static_cast<S*>(dhidden));
  return hipGetLastError();
}

int launch_logprob(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w,
                          const int32_t* target, const uint8_t* mask, int64_t T, int64_t H, int64_t V,
                          bool bf16, float* logp, float* lse, int32_t* status, void* ws, hipStream_t st) {
  return bf16 ? logprob_impl<BF16>(hidden, ld_hidden, w_head, ld_w, target, mask, T, H, V, logp, lse,
                                   status, ws, st)
              : logprob_impl<F32>(hidden, ld_hidden, w_head, ld_w, target, mask, T, H, V, logp, lse,
                                  status, ws, st);
}

int launch_backward(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w,
                           const int32_t* target, const float* lse, const float* g, int64_t T, int64_t H,
                           int64_t V, bool bf16, void* dhidden, float* dw, void* ws, hipStream_t st) {
  return bf16 ? backward_impl<BF16>(hidden, ld_hidden, w_head, ld_w, target, lse, g, T, H, V, dhidden, dw,
                                    ws, st)
              : backward_impl<F32>(hidden, ld_hidden, w_head, ld_w, target, lse, g, T, H, V, dhidden, dw,
                                   ws, st);
}

}  // namespace sao
