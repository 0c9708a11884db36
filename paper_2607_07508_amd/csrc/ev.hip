// Explained variance of the critic, EV = 1 - Var(R - V) / Var(R), the diagnostic
// of Sec. 4.4, over the loss-mask tokens.
//
// One pass over (values, ret, mask). Each thread keeps sums of its tokens shifted
// by its own first token (the shifted-data form of the variance, so a constant
// series gives exactly zero); threads, waves, blocks and calls are then combined
// with the pairwise update of Chan, Golub and LeVeque for (count, mean, sum of
// squared deviations), in a fixed order, so results do not depend on scheduling.
#include "common.hpp"
#include "launch.hpp"
#include "layout.hpp"
#include "reduce.hpp"

namespace sao {

// Count, means and sums of squared deviations of R and of d = R - V.
struct Moments {
  double n, mr, m2r, md, m2d;
};

// Pairwise combination of two disjoint sets' moments (a first, then b).
__device__ __forceinline__ Moments combine(const Moments& a, const Moments& b) {
  if (b.n == 0.0) return a;
  if (a.n == 0.0) return b;
  const double n = a.n + b.n;
  const double fb = b.n / n, cross = a.n * b.n / n;
  const double dr = b.mr - a.mr, dd = b.md - a.md;
  return {n, a.mr + dr * fb, a.m2r + b.m2r + dr * dr * cross, a.md + dd * fb, a.m2d + b.m2d + dd * dd * cross};
}

// Lane 0 gets the wave's moments, combined lane 0 first up to lane 63.
__device__ __forceinline__ Moments wave_combine(Moments m) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const Moments b{__shfl_down(m.n, o, 64), __shfl_down(m.mr, o, 64), __shfl_down(m.m2r, o, 64),
                    __shfl_down(m.md, o, 64), __shfl_down(m.m2d, o, 64)};
    if (lane < o) m = combine(m, b);
  }
  return m;
}

// Thread 0 gets the block's moments, combined wave 0 first.
template <int THREADS>
__device__ __forceinline__ Moments block_combine(Moments m) {
  __shared__ Moments sh[THREADS / 64];
  m = wave_combine(m);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    m = sh[0];
#pragma unroll
    for (int w = 1; w < THREADS / 64; ++w) m = combine(m, sh[w]);
  }
  return m;
}

// One thread's sums of its loss-mask tokens, shifted by its first one.
struct ShiftedSums {
  double kr = 0.0, kd = 0.0, n = 0.0, s1r = 0.0, s2r = 0.0, s1d = 0.0, s2d = 0.0;

  __device__ __forceinline__ void add(float v, float ret) {
    const double r = ret, d = r - static_cast<double>(v);
    if (n == 0.0) {
      kr = r;
      kd = d;
    }
    const double x = r - kr, y = d - kd;
    n += 1.0;
    s1r += x;
    s2r = fma(x, x, s2r);
    s1d += y;
    s2d = fma(y, y, s2d);
  }
  __device__ __forceinline__ Moments moments() const {
    if (n == 0.0) return {0.0, 0.0, 0.0, 0.0, 0.0};
    return {n, kr + s1r / n, fmax(0.0, s2r - s1r * s1r / n), kd + s1d / n, fmax(0.0, s2d - s1d * s1d / n)};
  }
};

__global__ __launch_bounds__(kLossThreads) void k_ev(const float* values, const float* ret, const uint8_t* mask,
                                                     int64_t T, Moments* part, bool vec_ok) {
  ShiftedSums acc;
  walk_tokens<kLossThreads>(
      T, vec_ok,
      [&](int64_t t) {
        const f32x4_t v4 = *reinterpret_cast<const f32x4_t*>(values + t);
        const f32x4_t r4 = *reinterpret_cast<const f32x4_t*>(ret + t);
        const uint32_t m4 = *reinterpret_cast<const uint32_t*>(mask + t);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (((m4 >> (8 * j)) & 0xffu) != 0) acc.add(v4[j], r4[j]);
      },
      [&](int64_t t) {
        if (mask[t] != 0) acc.add(values[t], ret[t]);
      });
  const Moments m = block_combine<kLossThreads>(acc.moments());
  if (threadIdx.x == 0) part[blockIdx.x] = m;
}

// Combines the block partials (thread i takes blocks i, i + THREADS, ... in
// order), then the caller's running moments first and this call's second; writes
// them back and, when asked, EV from them.
__global__ __launch_bounds__(kLossThreads) void k_ev_final(const Moments* part, int nblk, double* state,
                                                           double* ev) {
  Moments m{0.0, 0.0, 0.0, 0.0, 0.0};
  for (int i = threadIdx.x; i < nblk; i += kLossThreads) m = combine(m, part[i]);
  m = block_combine<kLossThreads>(m);
  if (threadIdx.x == 0) {
    const Moments s{state[0], state[1], state[2], state[3], state[4]};
    m = combine(s, m);
    state[0] = m.n;
    state[1] = m.mr;
    state[2] = m.m2r;
    state[3] = m.md;
    state[4] = m.m2d;
    if (ev) ev[0] = (m.n > 0.0 && m.m2r > 0.0) ? 1.0 - m.m2d / m.m2r : __builtin_nan("");
  }
}

int launch_explained_variance(const float* values, const float* ret, const uint8_t* mask, int64_t T,
                                     double* moments, double* ev, void* ws, hipStream_t st) {
  const EvLayout L = ev_layout(T);
  Moments* part = reinterpret_cast<Moments*>(static_cast<char*>(ws) + L.part);
  const int nblk = static_cast<int>(L.blocks);
  const bool vec_ok = ((reinterpret_cast<uintptr_t>(values) | reinterpret_cast<uintptr_t>(ret)) & 15u) == 0 &&
                      (reinterpret_cast<uintptr_t>(mask) & 3u) == 0;
  hipLaunchKernelGGL(k_ev, dim3(nblk), dim3(kLossThreads), 0, st, values, ret, mask, T, part, vec_ok);
  hipLaunchKernelGGL(k_ev_final, dim3(1), dim3(kLossThreads), 0, st, part, nblk, moments, ev);
  return hipGetLastError();
}

}  // namespace sao
