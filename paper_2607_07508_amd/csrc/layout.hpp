// Host-side workspace layouts shared by sao_workspace_size and the launchers.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace sao {

constexpr int64_t kTile = 256;
constexpr int64_t kRowsPerCountBlock = 1024;  // rows per block of the compaction count
constexpr int64_t kVocabBlock = 32768;        // vocabulary rows per backward dZ block (at least)
constexpr int64_t kVocabBlockMax = 65536;     // ... and at most
constexpr int kLossThreads = 256;
constexpr int kLossPerThread = 8;
constexpr int kLossMaxBlocks = 2048;

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline int64_t ceil_div(int64_t x, int64_t m) { return (x + m - 1) / m; }
inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

struct Carve {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  }
};

// sao_token_logprob
struct LogprobLayout {
  int64_t t_pad, n_count_blocks, m_tiles;
  size_t blk_counts, count, next, idx, hc, part, total;
};

inline LogprobLayout logprob_layout(int64_t T, int64_t H, int64_t V, size_t esize) {
  LogprobLayout L{};
  L.t_pad = round_up(T, kTile);
  L.n_count_blocks = ceil_div(T, kRowsPerCountBlock);
  L.m_tiles = ceil_div(V, kTile);
  Carve c;
  L.blk_counts = c.take(4 * static_cast<size_t>(L.n_count_blocks));
  L.count = c.take(4);
  L.next = c.take(4 * 8);  // the forward's tile counters, one per XCD
  L.idx = c.take(4 * static_cast<size_t>(L.t_pad));
  L.hc = c.take(esize * static_cast<size_t>(L.t_pad) * static_cast<size_t>(H));
  L.part = c.take(8 * static_cast<size_t>(L.m_tiles) * static_cast<size_t>(L.t_pad));
  L.total = c.off;
  return L;
}

// sao_loss_backward
struct BackwardLayout {
  int64_t t_pad, n_count_blocks, vc, n_vblocks;
  int dh_pieces;   // K pieces of the dH product (each with its own fp32 accumulator)
  size_t blk_counts, count, next, idx, pos, g_c, lse_c, y_c, hg, dh, dz, total;
};

// K pieces of the dH product: enough that its output tiles number at least 1024
// (four per CU) at the host bound of token rows, at most 8. Typically about a
// third of a chunk's rows carry a gradient, so this leaves a short chunk's dH
// launch with about one tile per CU.
constexpr int kMaxDhPieces = 8;
inline int dh_pieces(int64_t T, int64_t H) {
  const int64_t tiles = ceil_div(T, kTile) * ceil_div(H, kTile);
  int64_t p = ceil_div(1024, tiles);
  if (p < 1) p = 1;
  if (p > kMaxDhPieces) p = kMaxDhPieces;
  return static_cast<int>(p);
}

// MI355X's memory-side (Infinity) cache, shared by the XCDs, and its compute units.
constexpr int64_t kMemorySideCacheBytes = int64_t{256} << 20;
constexpr int64_t kGpuCus = 256;

inline int64_t gcd64(int64_t a, int64_t b) { return b == 0 ? a : gcd64(b, a % b); }

// Vocabulary rows per backward block. The target size is kVocabBlock, doubled up
// to kVocabBlockMax while one block's dz product would have fewer than 8192 tiles
// (32 per CU) at the host bound of token rows, so that short token chunks still
// give each launch many rounds of tiles and take fewer launches. V is then cut
// into as many blocks as that target size needs, as equal as possible.
// A block's dW product has (block tiles) x ceil(H / 256) output tiles, each as
// long as the whole token range, so a block whose dW tiles leave a partial last
// round idles part of the GPU for one long tile. Where the block's rows of W fit
// the memory-side cache, the block is therefore rounded up to a multiple of
// kGpuCus / gcd(kGpuCus, ceil(H / 256)) tiles (32 at H = 2048), which leaves
// only the last block with a partial round. (Measured: 1.4 % off c2's backward,
// 1.9 % off c3's.) Where the rounded-up block's rows of W would not fit the
// cache (H = 6144), the larger blocks slowed the logit recompute by more than
// dW gained; there the block is rounded down to that multiple instead (0.7 %
// off c4's backward).
inline int64_t vocab_block(int64_t t_pad, int64_t V, int64_t H, size_t esize) {
  int64_t vc = kVocabBlock;
  while (vc < kVocabBlockMax && (t_pad / kTile) * (vc / kTile) < 8192) vc *= 2;
  const int64_t blocks = ceil_div(V, vc);
  int64_t tiles = ceil_div(ceil_div(V, blocks), kTile);
  const int64_t align = kGpuCus / gcd64(kGpuCus, ceil_div(H, kTile));
  const int64_t rounded = round_up(tiles, align);
  if (blocks > 1 && rounded <= vc / kTile &&
      rounded * kTile * H * static_cast<int64_t>(esize) <= kMemorySideCacheBytes)
    tiles = rounded;
  else if (blocks > 1 && tiles >= align)
    tiles = tiles / align * align;
  return tiles * kTile;
}

inline BackwardLayout backward_layout(int64_t T, int64_t H, int64_t V, size_t esize) {
  BackwardLayout L{};
  L.t_pad = round_up(T, kTile);
  L.n_count_blocks = ceil_div(T, kRowsPerCountBlock);
  L.vc = vocab_block(L.t_pad, V, H, esize);
  L.n_vblocks = ceil_div(V, L.vc);
  L.dh_pieces = dh_pieces(T, H);
  Carve c;
  const size_t tp = static_cast<size_t>(L.t_pad);
  L.blk_counts = c.take(4 * static_cast<size_t>(L.n_count_blocks));
  L.count = c.take(4);
  L.next = c.take(4 * 8 * static_cast<size_t>(L.n_vblocks));  // the recompute's tile counters
  L.idx = c.take(4 * tp);
  L.pos = c.take(4 * static_cast<size_t>(T));
  L.g_c = c.take(4 * tp);
  L.lse_c = c.take(4 * tp);
  L.y_c = c.take(4 * tp);
  L.hg = c.take(esize * tp * static_cast<size_t>(H));
  L.dh = c.take(4 * tp * static_cast<size_t>(H) * static_cast<size_t>(L.dh_pieces));
  L.dz = c.take(esize * tp * static_cast<size_t>(L.vc));
  L.total = c.off;
  return L;
}

// Head of every advantage kernel's workspace: the int32 segments flag, then
// kCountSlots int64 slots that spread the loss-mask count's atomic adds (one
// slot per workgroup, modulo kCountSlots) before a one-block total.
constexpr int kCountSlots = 64;
struct SegHead {
  size_t bad, slots, total;
};
inline SegHead seg_head() {
  SegHead H{};
  Carve c;
  H.bad = c.take(4);
  H.slots = c.take(8 * kCountSlots);
  H.total = c.off;
  return H;
}

// sao_advantage needs only the head.
inline size_t advantage_workspace() { return seg_head().total; }

// sao_clipped_loss
struct LossLayout {
  int64_t blocks;
  size_t part_f, part_i, n_count, total;
};

inline LossLayout loss_layout(int64_t T) {
  LossLayout L{};
  int64_t blocks = ceil_div(T, static_cast<int64_t>(kLossThreads) * kLossPerThread);
  if (blocks > kLossMaxBlocks) blocks = kLossMaxBlocks;
  if (blocks < 1) blocks = 1;
  L.blocks = blocks;
  Carve c;
  L.part_f = c.take(16 * static_cast<size_t>(blocks));   // two doubles per block
  L.part_i = c.take(40 * static_cast<size_t>(blocks));   // five int64 per block
  L.n_count = c.take(8);
  L.total = c.off;
  return L;
}

// The largest sao_clipped_loss workspace (kLossMaxBlocks blocks; the three pieces
// are 256-byte multiples), the size of sao_clipped_loss_noalloc's static scratch.
// Every T fits, since the block count is capped.
constexpr size_t kLossScratchBytes = 16 * kLossMaxBlocks + 40 * kLossMaxBlocks + 256;
static_assert((16 * kLossMaxBlocks) % 256 == 0 && (40 * kLossMaxBlocks) % 256 == 0, "pieces stay aligned");

// sao_step_advantage: the head, then a step table of T entries (a trajectory's
// steps sit at its own token offset): start and end (int32), and two doubles
// (the step's value and reward, later its advantage and return).
struct StepLayout {
  size_t tab_a, tab_z, tab_v, tab_r, total;
};

inline StepLayout step_layout(int64_t T) {
  StepLayout L{};
  Carve c;
  c.take(seg_head().total);
  L.tab_a = c.take(4 * static_cast<size_t>(T));
  L.tab_z = c.take(4 * static_cast<size_t>(T));
  L.tab_v = c.take(8 * static_cast<size_t>(T));
  L.tab_r = c.take(8 * static_cast<size_t>(T));
  L.total = c.off;
  return L;
}

// sao_group_advantage / sao_running_mean_advantage need only the head.

// sao_ppo_loss shares the loss layout.

// sao_explained_variance: five doubles per block
struct EvLayout {
  int64_t blocks;
  size_t part, total;
};

inline EvLayout ev_layout(int64_t T) {
  EvLayout L{};
  L.blocks = loss_layout(T).blocks;
  Carve c;
  L.part = c.take(40 * static_cast<size_t>(L.blocks));
  L.total = c.off;
  return L;
}

// sao_value_loss (sao_value_forward needs none)
constexpr int kValueThreads = 256;
constexpr int64_t kValueRows = 128;           // rows per block of the value-loss pass
constexpr int64_t kValueCountBlocks = 1024;   // blocks of the mask count when N is not given

struct ValueLayout {
  int64_t row_blocks, count_blocks;
  size_t part_cnt, n_count, part_loss, part_dw, total;
};

inline ValueLayout value_layout(int64_t T, int64_t H) {
  ValueLayout L{};
  L.row_blocks = ceil_div(T, kValueRows);
  L.count_blocks = ceil_div(T, static_cast<int64_t>(kValueThreads) * 8);
  if (L.count_blocks > kValueCountBlocks) L.count_blocks = kValueCountBlocks;
  if (L.count_blocks < 1) L.count_blocks = 1;
  Carve c;
  L.part_cnt = c.take(8 * static_cast<size_t>(L.count_blocks));
  L.n_count = c.take(8);
  L.part_loss = c.take(8 * static_cast<size_t>(L.row_blocks));
  L.part_dw = c.take(4 * static_cast<size_t>(L.row_blocks) * static_cast<size_t>(H));
  L.total = c.off;
  return L;
}

}  // namespace sao
