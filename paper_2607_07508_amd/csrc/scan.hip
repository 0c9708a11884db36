// Skip-observation token-level GAE (Sec. 3.2, Eq. 4-5) as a segmented reverse scan.
//
// One workgroup per trajectory. Walking right to left, the state after a token is
//   s = (Vn, R, A, G): value of the next action, reward pending since the next
// action, and that action's advantage and return. Token t maps the state that
// enters from its right to the state that leaves to its left:
//   action (value v, reward r):  Vn' = v, R' = 0,
//                                A'  = (r + R) + gamma Vn - v + gamma lambda_b A,
//                                G'  = (r + R) + gamma G            (and A', G' are its outputs)
//   observation (reward r):      R' = R + r, everything else unchanged
// starting from s = 0 after the last token (no bootstrap after the last action;
// rewards before the first action leave through the left end and are dropped).
// Every such map, and every composition of them, has the form
//   Vn' = z Vn + cV,  R' = z R + cR,
//   A'  = cA + X (R + gamma Vn) + (kappa X + z) A,   kappa = gamma lambda_b,
//   G'  = cG + Y R + (gamma Y + z) G,
// where z = 1 for a run of observations only (then cV = cA = cG = X = Y = 0) and
// z = 0 once the run holds an action (then X = kappa^(n-1) and Y = gamma^(n-1) for
// its n actions). So a thread summarises its contiguous tokens by 7 numbers, the
// block scans the summaries (DPP lane moves inside each wave, then across waves
// through LDS), and each thread replays its tokens from the exact state that
// enters it. Arithmetic is float64. Tiles of 2048 tokens aligned to the global
// index give every thread 8 tokens that it reads and writes with 16-byte vector
// accesses.
#include "common.hpp"
#include "launch.hpp"
#include "layout.hpp"
#include "segments.hpp"

#include "../../include/sao.h"

namespace sao {

struct Aff {
  double z, cV, cR, X, cA, Y, cG;
};

__device__ __forceinline__ Aff aff_identity() { return Aff{1.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0}; }

// (F o G)(s) = F(G(s)). The coefficients of A and G in F are kappa F.X + F.z and
// gamma F.Y + F.z; products of them with G's come out in the same form.
__device__ __forceinline__ Aff compose(const Aff& F, const Aff& G, double gamma, double kappa) {
  const double fa = fma(kappa, F.X, F.z), fg = fma(gamma, F.Y, F.z);
  Aff r;
  r.z = F.z * G.z;
  r.cV = fma(F.z, G.cV, F.cV);
  r.cR = fma(F.z, G.cR, F.cR);
  r.X = fma(F.X, G.z, fa * G.X);
  r.cA = fma(F.X, fma(gamma, G.cV, G.cR), fma(fa, G.cA, F.cA));
  r.Y = fma(F.Y, G.z, fg * G.Y);
  r.cG = fma(F.Y, G.cR, fma(fg, G.cG, F.cG));
  return r;
}

// M o F for the map M of one token, F covering the tokens to its right
// (compose() with M's constants substituted: an action is z = 0, cV = v, cR = 0,
// X = Y = 1, cA = r - v, cG = r; an observation is the identity plus cR = r).
__device__ __forceinline__ void push_action(Aff& F, double v, double r, double gamma, double kappa) {
  const Aff G = F;
  F.z = 0.0;
  F.cV = v;
  F.cR = 0.0;
  F.X = fma(kappa, G.X, G.z);
  F.cA = fma(kappa, G.cA, fma(gamma, G.cV, G.cR + (r - v)));
  F.Y = fma(gamma, G.Y, G.z);
  F.cG = fma(gamma, G.cG, G.cR + r);
}
__device__ __forceinline__ void push_observation(Aff& F, double r) { F.cR += r; }

// A double moved across lanes by DPP (CTRL, ROW_MASK); lanes without a source keep `old`.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double old, double x) {
  const uint2 o = __builtin_bit_cast(uint2, old), v = __builtin_bit_cast(uint2, x);
  const int lo = __builtin_amdgcn_update_dpp(static_cast<int>(o.x), static_cast<int>(v.x), CTRL, ROW_MASK, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(static_cast<int>(o.y), static_cast<int>(v.y), CTRL, ROW_MASK, 0xf, false);
  return __builtin_bit_cast(double, make_uint2(static_cast<uint32_t>(lo), static_cast<uint32_t>(hi)));
}
// The map of another lane (identity where there is none).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ Aff dpp_aff(const Aff& x) {
  Aff o;
  o.z = dpp_f64<CTRL, ROW_MASK>(1.0, x.z);
  o.cV = dpp_f64<CTRL, ROW_MASK>(0.0, x.cV);
  o.cR = dpp_f64<CTRL, ROW_MASK>(0.0, x.cR);
  o.X = dpp_f64<CTRL, ROW_MASK>(0.0, x.X);
  o.cA = dpp_f64<CTRL, ROW_MASK>(0.0, x.cA);
  o.Y = dpp_f64<CTRL, ROW_MASK>(0.0, x.Y);
  o.cG = dpp_f64<CTRL, ROW_MASK>(0.0, x.cG);
  return o;
}

// Inclusive scan over the wave in lane order, S_l = F_l o F_{l-1} o ... o F_0:
// shifts by 1, 2, 4, 8 inside each row of 16 lanes (row_shr), then the last lane
// of row 0 into row 1 and of row 2 into row 3 (row_bcast:15), then lane 31 into
// rows 2 and 3 (row_bcast:31). DPP moves are VALU operations, so no step waits
// on the LDS crossbar.
__device__ __forceinline__ Aff wave_scan(Aff S, double gamma, double kappa) {
  S = compose(S, dpp_aff<0x111, 0xf>(S), gamma, kappa);
  S = compose(S, dpp_aff<0x112, 0xf>(S), gamma, kappa);
  S = compose(S, dpp_aff<0x114, 0xf>(S), gamma, kappa);
  S = compose(S, dpp_aff<0x118, 0xf>(S), gamma, kappa);
  S = compose(S, dpp_aff<0x142, 0xa>(S), gamma, kappa);
  S = compose(S, dpp_aff<0x143, 0xc>(S), gamma, kappa);
  return S;
}

constexpr int kScanThreads = 256;
constexpr int kScanPer = 8;                               // tokens per thread per tile
static_assert(kScanPer % 4 == 0, "whole blocks are read as 16-byte vectors");
constexpr int kScanTile = kScanThreads * kScanPer;        // tokens per tile

// State after applying map M to (Vn, R, A, G).
struct St {
  double Vn, R, A, G;
};
__device__ __forceinline__ St apply(const Aff& M, const St& s, double gamma, double kappa) {
  St o;
  o.Vn = fma(M.z, s.Vn, M.cV);
  o.R = fma(M.z, s.R, M.cR);
  o.A = fma(M.X, fma(gamma, s.Vn, s.R), fma(fma(kappa, M.X, M.z), s.A, M.cA));
  o.G = fma(M.Y, s.R, fma(fma(gamma, M.Y, M.z), s.G, M.cG));
  return o;
}

// One workgroup per trajectory. The trajectory is walked right to left in tiles
// of kScanTile tokens aligned to the global token index (so that each thread's
// kScanPer tokens are one aligned vector load per array); the state leaving a
// tile on the left enters the next tile from the right. Inside a tile each
// thread composes the maps of its tokens, the block scans the compositions,
// and each thread replays its tokens from the exact entering state.
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_advantage(
    const float* values, const float* rewards, const uint8_t* mask, const int32_t* cu, int32_t B,
    int64_t T, double gamma, double lam, double alpha, float* adv, float* ret, int64_t* slots,
    const int32_t* bad, bool vec_ok) {
  __shared__ Aff s_agg[2][kScanThreads / 64];  // alternate tiles use alternate halves
  __shared__ int64_t s_cnt[kScanThreads / 64];
  // The state entering the next tile from the right, double-buffered so that a
  // tile's writer never waits for the previous tile's readers.
  __shared__ St s_carry[2];
  // Each thread's values and rewards wait here, in its own slots, while the block
  // scans: holding them in registers instead would cost a wave per SIMD.
  __shared__ f32x4_t s_in[2 * kScanPer / 4][kScanThreads];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  if (*bad) {
    malformed_slice<kScanThreads, kCountSlots>(mask, B, T, adv, ret, nullptr, slots);
    return;
  }
  const int64_t s = cu[b], e = cu[b + 1];
  const int64_t L = e - s;
  if (L <= 0) return;
  double lam_b = lam;
  if (alpha > 0.0) {
    lam_b = 1.0 - 1.0 / (alpha * static_cast<double>(L));
    if (lam_b < 0.0) lam_b = 0.0;
  }
  const double kappa = gamma * lam_b;
  const int64_t first = s / kScanTile * kScanTile;           // aligned tile containing s
  int64_t total = 0;
  if (tid == 0) s_carry[0] = St{0.0, 0.0, 0.0, 0.0};         // nothing after the last token
  int buf = 0;
  // Thread i takes block 255 - i of each tile, so lane order runs right to left
  // and the reverse scan over tokens is a forward scan over lanes. Whole blocks
  // inside [s, e) use vector access (when the array bases allow it).
  for (int64_t t0 = (e - 1) / kScanTile * kScanTile; t0 >= first; t0 -= kScanTile) {
    const int64_t c0 = t0 + static_cast<int64_t>(kScanThreads - 1 - tid) * kScanPer;
    const bool full = vec_ok && c0 >= s && c0 + kScanPer <= e;
    float v[kScanPer], r[kScanPer];
    bool act[kScanPer];
    if (full) {
      const f32x4_t* pv = reinterpret_cast<const f32x4_t*>(values + c0);
      const f32x4_t* pr = reinterpret_cast<const f32x4_t*>(rewards + c0);
      const uint32_t* pm = reinterpret_cast<const uint32_t*>(mask + c0);
#pragma unroll
      for (int q = 0; q < kScanPer / 4; ++q) {
        const f32x4_t vq = pv[q], rq = pr[q];
        const uint32_t mq = pm[q];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v[4 * q + j] = vq[j];
          r[4 * q + j] = rq[j];
          act[4 * q + j] = ((mq >> (8 * j)) & 0xffu) != 0;
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < kScanPer; ++j) {
        const int64_t t = c0 + j;
        const bool in = t >= s && t < e;
        v[j] = in ? values[t] : 0.0f;
        r[j] = in ? rewards[t] : 0.0f;
        act[j] = in && mask[t] != 0;
      }
    }
#pragma unroll
    for (int q = 0; q < kScanPer / 4; ++q) {
      s_in[q][tid] = f32x4_t{v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
      s_in[kScanPer / 4 + q][tid] = f32x4_t{r[4 * q], r[4 * q + 1], r[4 * q + 2], r[4 * q + 3]};
    }
    // Pass 1: this thread's tokens as one map (tokens outside [s, e) are identities).
    Aff F = aff_identity();
    int64_t cnt = 0;
#pragma unroll
    for (int j = kScanPer - 1; j >= 0; --j) {
      const bool in = full || (c0 + j >= s && c0 + j < e);
      if (!in) continue;
      if (act[j]) {
        ++cnt;
        push_action(F, v[j], r[j], gamma, kappa);
      } else {
        push_observation(F, r[j]);
      }
    }
    total += cnt;
    const Aff S = wave_scan(F, gamma, kappa);                     // this lane and the lanes to its right
    const Aff E = dpp_aff<0x138, 0xf>(S);          // wave_shr:1, the lanes to its right only
    // One barrier per tile: the half of s_agg written here was last read two tiles
    // ago, and the carry written at the end of the previous tile is published by it.
    if (lane == 63) s_agg[buf][wave] = S;
    __syncthreads();
    // State entering this wave: the carry through the waves to its right (lower waves).
    St sw = s_carry[buf];
    for (int w = 0; w < wave; ++w) sw = apply(s_agg[buf][w], sw, gamma, kappa);
    St st = apply(E, sw, gamma, kappa);
    // Pass 2: replay the tokens from that state and write the outputs.
#pragma unroll
    for (int q = 0; q < kScanPer / 4; ++q) {
      const f32x4_t vq = s_in[q][tid], rq = s_in[kScanPer / 4 + q][tid];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[4 * q + j] = vq[j];
        r[4 * q + j] = rq[j];
      }
    }
    float oa[kScanPer], og[kScanPer];
#pragma unroll
    for (int j = kScanPer - 1; j >= 0; --j) {
      oa[j] = 0.0f;
      og[j] = 0.0f;
      const bool in = full || (c0 + j >= s && c0 + j < e);
      if (!in) continue;
      const double rr = r[j];
      if (act[j]) {
        const double vv = v[j];
        const double rt = rr + st.R;
        const double An = fma(kappa, st.A, fma(gamma, st.Vn, rt - vv));
        const double Gn = fma(gamma, st.G, rt);
        oa[j] = static_cast<float>(An);
        og[j] = static_cast<float>(Gn);
        st.Vn = vv;
        st.R = 0.0;
        st.A = An;
        st.G = Gn;
      } else {
        st.R += rr;
      }
    }
    if (full) {
      f32x4_t* qa = reinterpret_cast<f32x4_t*>(adv + c0);
      f32x4_t* qg = reinterpret_cast<f32x4_t*>(ret + c0);
#pragma unroll
      for (int q = 0; q < kScanPer / 4; ++q) {
        qa[q] = f32x4_t{oa[4 * q], oa[4 * q + 1], oa[4 * q + 2], oa[4 * q + 3]};
        qg[q] = f32x4_t{og[4 * q], og[4 * q + 1], og[4 * q + 2], og[4 * q + 3]};
      }
    } else {
#pragma unroll
      for (int j = 0; j < kScanPer; ++j) {
        const int64_t t = c0 + j;
        if (t >= s && t < e) {
          adv[t] = oa[j];
          ret[t] = og[j];
        }
      }
    }
    // The state leaving this tile on the left (the last thread's final state) enters
    // the next tile; the other buffer's readers finished before this tile's barrier.
    buf ^= 1;
    if (tid == kScanThreads - 1) s_carry[buf] = st;
  }
  const int64_t wcnt = wave_sum(total);
  __syncthreads();
  if (lane == 0) s_cnt[wave] = wcnt;
  __syncthreads();
  if (tid == 0) {
    int64_t tot = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) tot += s_cnt[w];
    add_count<kCountSlots>(slots, tot);
  }
}

int launch_advantage(const float* values, const float* rewards, const uint8_t* mask,
                            const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma, double lam,
                            double alpha, float* adv, float* ret, int64_t* n_tokens, int32_t* status,
                            void* ws, hipStream_t st) {
  const SegHead H = seg_head();
  char* w8 = static_cast<char*>(ws);
  int32_t* bad = reinterpret_cast<int32_t*>(w8 + H.bad);
  int64_t* slots = reinterpret_cast<int64_t*>(w8 + H.slots);
  hipLaunchKernelGGL((k_check_segments<256, kCountSlots>), dim3(1), dim3(256), 0, st, cu_seqlens, B, T, bad, slots,
                     status);
  // Vector access needs 16-byte aligned float arrays and an 8-byte aligned mask.
  const uintptr_t f = reinterpret_cast<uintptr_t>(values) | reinterpret_cast<uintptr_t>(rewards) |
                      reinterpret_cast<uintptr_t>(adv) | reinterpret_cast<uintptr_t>(ret);
  const bool vec_ok = (f & 15u) == 0 && (reinterpret_cast<uintptr_t>(mask) & 7u) == 0;
  hipLaunchKernelGGL(k_advantage, dim3(B), dim3(kScanThreads), 0, st, values, rewards, mask, cu_seqlens,
                     B, T, gamma, lam, alpha, adv, ret, slots, bad, vec_ok);
  if (n_tokens) hipLaunchKernelGGL(k_slots_total<kCountSlots>, dim3(1), dim3(64), 0, st, slots, n_tokens);
  return hipGetLastError();
}

}  // namespace sao
