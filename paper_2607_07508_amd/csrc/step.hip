// Step-level GAE (App. A.1): one advantage per agentic step.
//
// A step is a maximal run of loss-mask tokens inside a trajectory (one model
// turn). With steps [a_i, z_i), i < n, and a_n = the trajectory's end:
//   V_i = mean of values[a_i .. z_i)  or  values[z_i - 1]      (step average / last token)
//   R_i = sum of rewards[a_i .. a_{i+1})                       (observations fold into the step)
//   A_i = R_i + gamma V_{i+1} - V_i + gamma lambda_b A_{i+1},  G_i = R_i + gamma G_{i+1}
// with V_n = A_n = G_n = 0 and lambda_b = 1 - 1/(alpha n) when alpha > 0.
//
// One workgroup per trajectory, three phases separated by barriers:
//  1. left to right over 2048-token tiles: each token's step starts a new
//     segment (a step's run and the observations after it); a block scan numbers
//     the steps and a segmented block scan sums values (on the run) and rewards
//     (over the segment), with the open segment's sums carried from tile to tile.
//     Each step's start, end and sums (or last value) go to a per-trajectory
//     table in the workspace, written once, by the thread holding the token;
//  2. the recurrence over steps: each thread takes a contiguous chunk of steps,
//     summarises it as an affine map of the state entering from its right, one
//     thread chains the chunk maps, and each thread replays its chunk;
//  3. each wave writes its steps' tokens: A_i and G_i on the run, zeros on the
//     observations after it, and the step's last token in `last`.
// Arithmetic is float64; every reduction runs in a fixed order.
#include "common.hpp"
#include "launch.hpp"
#include "layout.hpp"
#include "segments.hpp"

namespace sao {

constexpr int kStepThreads = 256;
constexpr int kStepPer = 8;                               // tokens per thread per tile
constexpr int kStepTile = kStepThreads * kStepPer;

namespace {
// Lane moves by DPP (CTRL, ROW_MASK): VALU operations, no LDS crossbar. Lanes
// without a source, and rows outside ROW_MASK, keep `old`. A wave's inclusive
// scan in lane order takes row_shr 1, 2, 4, 8 (0x111..0x118, all rows), then
// row_bcast:15 (0x142, rows 1 and 3) and row_bcast:31 (0x143, rows 2 and 3);
// wave_shr:1 (0x138) turns it into the exclusive one.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_i32(int old, int x) {
  return __builtin_amdgcn_update_dpp(old, x, CTRL, ROW_MASK, 0xf, false);
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double old, double x) {
  const uint2 o = __builtin_bit_cast(uint2, old), v = __builtin_bit_cast(uint2, x);
  return __builtin_bit_cast(double, make_uint2(static_cast<uint32_t>(dpp_i32<CTRL, ROW_MASK>(static_cast<int>(o.x), static_cast<int>(v.x))),
                                               static_cast<uint32_t>(dpp_i32<CTRL, ROW_MASK>(static_cast<int>(o.y), static_cast<int>(v.y)))));
}
}  // namespace

// Sums of a segmented scan: n counts the segments that start inside the span; if
// there are any, v and r cover only the part after the last start.
struct Seg {
  int n;
  double v, r;
};
// x then y (x on the left).
__device__ __forceinline__ Seg seg_combine(const Seg& x, const Seg& y) {
  return y.n ? Seg{x.n + y.n, y.v, y.r} : Seg{x.n, x.v + y.v, x.r + y.r};
}
// The sums of another lane (the empty sums where there is none).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ Seg dpp_seg(const Seg& x) {
  return Seg{dpp_i32<CTRL, ROW_MASK>(0, x.n), dpp_f64<CTRL, ROW_MASK>(0.0, x.v), dpp_f64<CTRL, ROW_MASK>(0.0, x.r)};
}

// Exclusive segmented scan over the block in thread order, the sums `carry`
// standing before thread 0; returns the sums entering this thread, with n the
// starts before it in this call. `out` gets everything (carry's sums included,
// n = the call's starts) for the next call. Successive calls alternate between
// the two halves of `sh`, so no call waits for the previous one's readers.
__device__ __forceinline__ Seg block_segmented_scan(const Seg& x, const Seg& carry, Seg* sh, Seg* out) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  Seg incl = x;  // the empty sums on the left change nothing
  incl = seg_combine(dpp_seg<0x111, 0xf>(incl), incl);
  incl = seg_combine(dpp_seg<0x112, 0xf>(incl), incl);
  incl = seg_combine(dpp_seg<0x114, 0xf>(incl), incl);
  incl = seg_combine(dpp_seg<0x118, 0xf>(incl), incl);
  incl = seg_combine(dpp_seg<0x142, 0xa>(incl), incl);
  incl = seg_combine(dpp_seg<0x143, 0xc>(incl), incl);
  const Seg excl = dpp_seg<0x138, 0xf>(incl);
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  Seg before{0, carry.v, carry.r};
  for (int w = 0; w < wave; ++w) before = seg_combine(before, sh[w]);
  Seg all = before;
  for (int w = wave; w < kStepThreads / 64; ++w) all = seg_combine(all, sh[w]);
  *out = all;
  return seg_combine(before, excl);
}

__global__ __launch_bounds__(kStepThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_step_advantage(
    const float* values, const float* rewards, const uint8_t* mask, const int32_t* cu, int32_t B, int64_t T,
    double gamma, double lam, double alpha, bool last_value, float* adv, float* ret, uint8_t* last,
    int64_t* slots, const int32_t* bad, int32_t* tab_a, int32_t* tab_z, double* tab_v, double* tab_r,
    bool vec_ok, bool out_vec) {
  __shared__ Seg s_seg[2][kStepThreads / 64];  // alternate tiles use alternate halves
  __shared__ double s_map[kStepThreads][4];   // per chunk: A = cA + mA A_in, G = cG + mG G_in
  __shared__ double s_in[kStepThreads][2];    // (A, G) entering each chunk from the right
  __shared__ int64_t s_cnt[kStepThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  if (*bad) {
    malformed_slice<kStepThreads, kCountSlots>(mask, B, T, adv, ret, last, slots);
    return;
  }
  const int64_t s = cu[b], e = cu[b + 1];
  const int64_t L = e - s;
  if (L <= 0) return;
  // The step table of this trajectory: entries [0, n) at offset s (n <= L).
  int32_t* ta = tab_a + s;
  int32_t* tz = tab_z + s;
  double* tv = tab_v + s;
  double* tr = tab_r + s;

  // Phase 1: step starts, ends and sums (segment i: step i's run and the
  // observations after it, up to the next step; rewards before the first step
  // fall in no segment).
  int n = 0;
  Seg carry{0, 0.0, 0.0};
  int64_t cnt = 0;
  int tile = 0;
  for (int64_t t0 = s / kStepTile * kStepTile; t0 < e; t0 += kStepTile, ++tile) {
    const int64_t c0 = t0 + static_cast<int64_t>(tid) * kStepPer;
    bool m[kStepPer + 2];  // m[j] is token c0 - 1 + j
    float v[kStepPer], r[kStepPer];  // v is 0 off the runs
    m[0] = c0 - 1 >= s && c0 - 1 < e && mask[c0 - 1] != 0;
    m[kStepPer + 1] = c0 + kStepPer >= s && c0 + kStepPer < e && mask[c0 + kStepPer] != 0;
    if (vec_ok && c0 >= s && c0 + kStepPer <= e) {
      const f32x4_t* pv = reinterpret_cast<const f32x4_t*>(values + c0);
      const f32x4_t* pr = reinterpret_cast<const f32x4_t*>(rewards + c0);
      const uint64_t m8 = *reinterpret_cast<const uint64_t*>(mask + c0);
#pragma unroll
      for (int q = 0; q < kStepPer / 4; ++q) {
        const f32x4_t vq = pv[q], rq = pr[q];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int k = 4 * q + j;
          m[k + 1] = ((m8 >> (8 * k)) & 0xffu) != 0;
          v[k] = m[k + 1] ? vq[j] : 0.0f;
          r[k] = rq[j];
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < kStepPer; ++j) {
        const int64_t t = c0 + j;
        const bool in = t >= s && t < e;
        m[j + 1] = in && mask[t] != 0;
        v[j] = m[j + 1] ? values[t] : 0.0f;
        r[j] = in ? rewards[t] : 0.0f;
      }
    }
    // This thread's starts, and its sums after its last start.
    int ns = 0;
    Seg x{0, 0.0, 0.0};
#pragma unroll
    for (int j = 0; j < kStepPer; ++j) {
      const bool st = m[j + 1] && !m[j];
      cnt += m[j + 1] ? 1 : 0;
      ns += st ? 1 : 0;
      if (st) x = Seg{0, 0.0, 0.0};
      x.v += static_cast<double>(v[j]);
      x.r += static_cast<double>(r[j]);
    }
    x.n = ns;
    Seg next_carry;
    Seg run = block_segmented_scan(x, carry, s_seg[tile & 1], &next_carry);
    const int first = n + run.n, tot_s = next_carry.n;
    // Replay: `key` is the step whose segment holds the token (-1 before the first).
    int key = first - 1;
#pragma unroll
    for (int j = 0; j < kStepPer; ++j) {
      const int64_t t = c0 + j;
      if (t < s || t >= e) continue;
      const int32_t off = static_cast<int32_t>(t - s);
      if (m[j + 1] && !m[j]) {
        ++key;
        run = Seg{1, 0.0, 0.0};
        ta[key] = off;
      }
      run.v += static_cast<double>(v[j]);
      run.r += static_cast<double>(r[j]);
      if (key < 0) continue;
      if (m[j + 1] && !m[j + 2]) {
        tz[key] = off + 1;
        if (last_value) tv[key] = static_cast<double>(v[j]);
      }
      const bool seg_end = t == e - 1 || (m[j + 2] && !m[j + 1]);
      if (seg_end) {
        if (!last_value) tv[key] = run.v;
        tr[key] = run.r;
      }
    }
    n += tot_s;
    carry = next_carry;
  }
  __syncthreads();  // the table is written

  // Phase 2: A_i and G_i. Thread j takes steps [p, q); its map sends the state
  // (A_q, G_q) entering from the right to (A_p, G_p). The table then holds them.
  double lam_b = lam;
  if (alpha > 0.0) {
    lam_b = 1.0 - 1.0 / (alpha * static_cast<double>(n));
    if (lam_b < 0.0) lam_b = 0.0;
  }
  const double kappa = gamma * lam_b;
  const int per = (n + kStepThreads - 1) / kStepThreads;
  const int p = min(n, tid * per), q = min(n, p + per);
  auto step_value = [&](int i) {
    return last_value ? tv[i] : tv[i] / static_cast<double>(tz[i] - ta[i]);
  };
  const double v_right = q < n ? step_value(q) : 0.0;   // read before any thread overwrites the table
  {
    double cA = 0.0, mA = 1.0, cG = 0.0, mG = 1.0, vn = v_right;
    for (int i = q - 1; i >= p; --i) {
      const double vi = step_value(i), ri = tr[i];
      cA = fma(kappa, cA, fma(gamma, vn, ri - vi));
      mA *= kappa;
      cG = fma(gamma, cG, ri);
      mG *= gamma;
      vn = vi;
    }
    s_map[tid][0] = cA;
    s_map[tid][1] = mA;
    s_map[tid][2] = cG;
    s_map[tid][3] = mG;
  }
  __syncthreads();
  if (tid == 0) {
    double A = 0.0, G = 0.0;
    const int chunks = per > 0 ? (n + per - 1) / per : 0;
    for (int j = chunks - 1; j >= 0; --j) {
      s_in[j][0] = A;
      s_in[j][1] = G;
      A = fma(s_map[j][1], A, s_map[j][0]);
      G = fma(s_map[j][3], G, s_map[j][2]);
    }
  }
  __syncthreads();
  if (p < q) {
    double A = s_in[tid][0], G = s_in[tid][1], vn = v_right;
    for (int i = q - 1; i >= p; --i) {
      const double vi = step_value(i), ri = tr[i];
      A = fma(kappa, A, fma(gamma, vn, ri - vi));
      G = fma(gamma, G, ri);
      vn = vi;
      tv[i] = A;
      tr[i] = G;
    }
  }
  __syncthreads();

  // Phase 3: outputs. Tokens before the first step, and every token of a
  // trajectory without steps, are zero; each wave then writes its steps' spans.
  const int64_t head = n > 0 ? ta[0] : L;
  for (int64_t t = tid; t < head; t += kStepThreads) {
    adv[s + t] = 0.0f;
    ret[s + t] = 0.0f;
    if (last) last[s + t] = 0;
  }
  for (int i = wave; i < n; i += kStepThreads / 64) {
    const int64_t a = s + ta[i], z = s + tz[i], nxt = s + (i + 1 < n ? ta[i + 1] : L);  // global indices
    const float A = static_cast<float>(tv[i]), G = static_cast<float>(tr[i]);
    auto one = [&](int64_t t) {
      const bool in = t < z;
      adv[t] = in ? A : 0.0f;
      ret[t] = in ? G : 0.0f;
      if (last) last[t] = t == z - 1 ? 1 : 0;
    };
    // The span's 4-aligned interior with 16-byte stores (4-byte ones for `last`),
    // its edges token by token.
    const int64_t b0 = out_vec ? min(nxt, (a + 3) / 4 * 4) : nxt;
    const int64_t b1 = out_vec ? max(b0, nxt / 4 * 4) : nxt;
    for (int64_t t = a + lane; t < b0; t += 64) one(t);
    for (int64_t t = b0 + 4 * static_cast<int64_t>(lane); t < b1; t += 4 * 64) {
      const bool i0 = t < z, i1 = t + 1 < z, i2 = t + 2 < z, i3 = t + 3 < z;
      *reinterpret_cast<f32x4_t*>(adv + t) = f32x4_t{i0 ? A : 0.0f, i1 ? A : 0.0f, i2 ? A : 0.0f, i3 ? A : 0.0f};
      *reinterpret_cast<f32x4_t*>(ret + t) = f32x4_t{i0 ? G : 0.0f, i1 ? G : 0.0f, i2 ? G : 0.0f, i3 ? G : 0.0f};
      if (last) {
        const int64_t k = z - 1 - t;  // byte k of this block is the step's last token
        *reinterpret_cast<uint32_t*>(last + t) = (k >= 0 && k < 4) ? (1u << (8 * k)) : 0u;
      }
    }
    for (int64_t t = b1 + lane; t < nxt; t += 64) one(t);
  }

  const int64_t wcnt = wave_sum(cnt);
  __syncthreads();
  if (lane == 0) s_cnt[wave] = wcnt;
  __syncthreads();
  if (tid == 0) {
    int64_t tot = 0;
    for (int w = 0; w < kStepThreads / 64; ++w) tot += s_cnt[w];
    add_count<kCountSlots>(slots, tot);
  }
}

int launch_step_advantage(const float* values, const float* rewards, const uint8_t* mask,
                                 const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma, double lam,
                                 double alpha, bool last_value, float* adv, float* ret, uint8_t* last,
                                 int64_t* n_tokens, int32_t* status, void* ws, hipStream_t st) {
  const StepLayout Ly = step_layout(T);
  char* w8 = static_cast<char*>(ws);
  const SegHead H = seg_head();
  int32_t* bad = reinterpret_cast<int32_t*>(w8 + H.bad);
  int64_t* slots = reinterpret_cast<int64_t*>(w8 + H.slots);
  hipLaunchKernelGGL((k_check_segments<256, kCountSlots>), dim3(1), dim3(256), 0, st, cu_seqlens, B, T, bad, slots,
                     status);
  // Whole in-trajectory blocks of 8 tokens use vector loads when the bases allow them.
  const bool vec_ok = ((reinterpret_cast<uintptr_t>(values) | reinterpret_cast<uintptr_t>(rewards)) & 15u) == 0 &&
                      (reinterpret_cast<uintptr_t>(mask) & 7u) == 0;
  // The output spans use 16-byte stores when adv and ret are 16-byte aligned and `last` (if given) 4-byte aligned.
  const bool out_vec = ((reinterpret_cast<uintptr_t>(adv) | reinterpret_cast<uintptr_t>(ret)) & 15u) == 0 &&
                       (reinterpret_cast<uintptr_t>(last) & 3u) == 0;
  hipLaunchKernelGGL(k_step_advantage, dim3(B), dim3(kStepThreads), 0, st, values, rewards, mask, cu_seqlens, B, T,
                     gamma, lam, alpha, last_value, adv, ret, last, slots, bad,
                     reinterpret_cast<int32_t*>(w8 + Ly.tab_a), reinterpret_cast<int32_t*>(w8 + Ly.tab_z),
                     reinterpret_cast<double*>(w8 + Ly.tab_v), reinterpret_cast<double*>(w8 + Ly.tab_r), vec_ok,
                     out_vec);
  if (n_tokens) hipLaunchKernelGGL(k_slots_total<kCountSlots>, dim3(1), dim3(64), 0, st, slots, n_tokens);
  return hipGetLastError();
}

}  // namespace sao
