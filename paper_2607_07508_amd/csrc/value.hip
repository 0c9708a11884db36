// Critic head of the PPO-style update (Sec. 2): a bias-free H -> 1 projection of
// the hidden states and its squared-error loss against the lambda = 1 returns,
//   v_t = h_t . w_v,   L_V = (1/N) sum_t m_t (v_t - G_t)^2,
//   dv_t = 2 m_t (v_t - G_t) / N,  dH_v[t] = dv_t w_v,  dw_v += sum_t dv_t h_t.
// Both passes stream the hidden states once (HBM-bound). The weight gradient is
// reduced as per-row-block partials followed by a fixed-order column sum, and
// the loss as per-row-block float64 partials, so results are deterministic.
#include "common.hpp"
#include "launch.hpp"
#include "layout.hpp"
#include "reduce.hpp"

namespace sao {

// Widen one 16-byte chunk to floats.
__device__ __forceinline__ void widen(const v4u& x, float (&f)[8], BF16) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(x[i] << 16);
    f[2 * i + 1] = __uint_as_float(x[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void widen(const v4u& x, float (&f)[4], F32) {
#pragma unroll
  for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(x[i]);
}
__device__ __forceinline__ v4u narrow(const float (&f)[8], BF16) {
  v4u x;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    x[i] = pack_bf16x2(f[2 * i], f[2 * i + 1]);
  return x;
}
__device__ __forceinline__ v4u narrow(const float (&f)[4], F32) {
  return v4u{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3])};
}

// One wave per row: v[t] = hidden[t] . w_v.
template <class E>
__global__ __launch_bounds__(kValueThreads) void k_value_forward(const typename E::storage* hidden, int64_t ld,
                                                                 const typename E::storage* w, int64_t T,
                                                                 int64_t H, float* v) {
  constexpr int P = E::kPerChunk;
  const int lane = threadIdx.x & 63;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * (kValueThreads / 64) + (threadIdx.x >> 6);
  if (t >= T) return;
  const v4u* row = reinterpret_cast<const v4u*>(hidden + t * ld);
  const v4u* wv = reinterpret_cast<const v4u*>(w);
  const int64_t chunks = H / P;
  float acc = 0.0f;
  for (int64_t c = lane; c < chunks; c += 64) {
    float h[P], x[P];
    widen(row[c], h, E{});
    widen(wv[c], x, E{});
#pragma unroll
    for (int e = 0; e < P; ++e) acc = fmaf(h[e], x[e], acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) v[t] = acc;
}

// Block (row block rb, chunk block cb): dv for kValueRows rows, dH_v for those
// rows over 256 chunks of H, the partial dw_v of those rows, and (cb == 0) the
// row block's float64 loss partial.
template <class E>
__global__ __launch_bounds__(kValueThreads) void k_value_rows(
    const typename E::storage* hidden, int64_t ld, const typename E::storage* w, const float* v,
    const float* ret, const uint8_t* mask, int64_t T, int64_t H, const int64_t* n_ptr,
    typename E::storage* dhidden, double* part_loss, float* part_dw) {
  constexpr int P = E::kPerChunk;
  __shared__ float s_dv[kValueRows];
  __shared__ double s_red[kValueThreads / 64];
  const int tid = threadIdx.x;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kValueRows;
  const int nrows = static_cast<int>(T - r0 < kValueRows ? T - r0 : kValueRows);
  const int64_t N = *n_ptr;
  const double invN = N > 0 ? 1.0 / static_cast<double>(N) : 0.0;
  double l = 0.0;
  if (tid < kValueRows) {
    float dv = 0.0f;
    if (tid < nrows && N > 0 && mask[r0 + tid] != 0) {
      const double d = static_cast<double>(v[r0 + tid]) - static_cast<double>(ret[r0 + tid]);
      l = d * d;
      dv = static_cast<float>(2.0 * d * invN);
    }
    s_dv[tid] = dv;
  }
  if (blockIdx.y == 0) {  // uniform over the block
    l = block_sum<kValueThreads>(l, s_red);
    if (tid == 0) part_loss[blockIdx.x] = l;
  }
  __syncthreads();
  const int64_t c = static_cast<int64_t>(blockIdx.y) * kValueThreads + tid;
  if (c >= H / P) return;
  float wf[P], acc[P];
  widen(reinterpret_cast<const v4u*>(w)[c], wf, E{});
#pragma unroll
  for (int e = 0; e < P; ++e) acc[e] = 0.0f;
  // Rows in groups of four: the four rows' hidden chunks are loaded before any
  // is used, so that four loads are in flight per thread (rows with dv = 0 are
  // not read; their dH_v chunk is zero).
  for (int i0 = 0; i0 < nrows; i0 += 4) {
    v4u hr[4];
    float dd[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      dd[u] = i0 + u < nrows ? s_dv[i0 + u] : 0.0f;
      if (dd[u] != 0.0f)  // uniform over the block
        hr[u] = reinterpret_cast<const v4u*>(hidden + (r0 + i0 + u) * ld)[c];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (i0 + u >= nrows) break;
      const float d = dd[u];
      float o[P];
#pragma unroll
      for (int e = 0; e < P; ++e) o[e] = d == 0.0f ? 0.0f : d * wf[e];
      reinterpret_cast<v4u*>(dhidden + (r0 + i0 + u) * H)[c] = narrow(o, E{});
      if (d != 0.0f) {
        float h[P];
        widen(hr[u], h, E{});
#pragma unroll
        for (int e = 0; e < P; ++e) acc[e] = fmaf(d, h[e], acc[e]);
      }
    }
  }
  float* out = part_dw + static_cast<int64_t>(blockIdx.x) * H + c * P;
#pragma unroll
  for (int e = 0; e < P; ++e) out[e] = acc[e];
}

// dw_v[col] += sum over row blocks; block 0 also adds the loss. A block takes
// 64 columns: wave w sums row blocks w, w + 4, w + 8, ... into 8 partial sums
// per lane (so that 8 loads are in flight), which it combines in a fixed order;
// then the 4 waves' sums are added in wave order. Every run adds in the same
// order, so the result is deterministic.
__global__ __launch_bounds__(kValueThreads) void k_value_final(const float* part_dw, const double* part_loss,
                                                               int64_t row_blocks, int64_t H,
                                                               const int64_t* n_ptr, double* loss_v,
                                                               float* dw_v) {
  constexpr int kWaves = kValueThreads / 64;
  constexpr int kLanes = 8;
  __shared__ double s_red[kWaves];
  __shared__ float s_col[kWaves][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (blockIdx.x == 0) {  // uniform over the block
    double l = 0.0;
    for (int64_t i = threadIdx.x; i < row_blocks; i += kValueThreads) l += part_loss[i];
    l = block_sum<kValueThreads>(l, s_red);
    const int64_t N = *n_ptr;
    if (threadIdx.x == 0 && N > 0) loss_v[0] += l / static_cast<double>(N);
  }
  const int64_t col = static_cast<int64_t>(blockIdx.x) * 64 + lane;
  float acc[kLanes];
#pragma unroll
  for (int u = 0; u < kLanes; ++u) acc[u] = 0.0f;
  if (col < H) {
    int64_t rb = wave;
    for (; rb + (kLanes - 1) * kWaves < row_blocks; rb += kLanes * kWaves) {
#pragma unroll
      for (int u = 0; u < kLanes; ++u) acc[u] += part_dw[(rb + u * kWaves) * H + col];
    }
    // fewer than kLanes row blocks of this wave remain
#pragma unroll
    for (int u = 0; u < kLanes; ++u)
      if (rb + u * kWaves < row_blocks) acc[u] += part_dw[(rb + u * kWaves) * H + col];
  }
  s_col[wave][lane] = ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
  __syncthreads();
  if (wave == 0 && col < H) {
    float t = s_col[0][lane];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) t += s_col[w][lane];
    dw_v[col] += t;
  }
}

int launch_value_forward(const void* hidden, int64_t ld_hidden, const void* w_v, int64_t T, int64_t H,
                                bool bf16, float* v, hipStream_t st) {
  const dim3 grid(static_cast<unsigned>(ceil_div(T, kValueThreads / 64)));
  if (bf16)
    hipLaunchKernelGGL(k_value_forward<BF16>, grid, dim3(kValueThreads), 0, st,
                       static_cast<const uint16_t*>(hidden), ld_hidden, static_cast<const uint16_t*>(w_v), T, H, v);
  else
    hipLaunchKernelGGL(k_value_forward<F32>, grid, dim3(kValueThreads), 0, st, static_cast<const float*>(hidden),
                       ld_hidden, static_cast<const float*>(w_v), T, H, v);
  return hipGetLastError();
}

int launch_value_loss(const void* hidden, int64_t ld_hidden, const void* w_v, const float* v,
                             const float* ret, const uint8_t* mask, int64_t T, int64_t H, const int64_t* n_tokens,
                             bool bf16, double* loss_v, void* dhidden_v, float* dw_v, void* ws, hipStream_t st) {
  const ValueLayout L = value_layout(T, H);
  char* w8 = static_cast<char*>(ws);
  const int64_t* n_ptr = n_tokens;
  if (!n_ptr) {
    int64_t* part = reinterpret_cast<int64_t*>(w8 + L.part_cnt);
    int64_t* total = reinterpret_cast<int64_t*>(w8 + L.n_count);
    const int nblk = static_cast<int>(L.count_blocks);
    hipLaunchKernelGGL(k_mask_count<kValueThreads>, dim3(nblk), dim3(kValueThreads), 0, st, mask, T, part);
    hipLaunchKernelGGL(k_count_total<kValueThreads>, dim3(1), dim3(kValueThreads), 0, st, part, nblk, total);
    n_ptr = total;
  }
  double* part_loss = reinterpret_cast<double*>(w8 + L.part_loss);
  float* part_dw = reinterpret_cast<float*>(w8 + L.part_dw);
  const int P = bf16 ? BF16::kPerChunk : F32::kPerChunk;
  const dim3 grid(static_cast<unsigned>(L.row_blocks), static_cast<unsigned>(ceil_div(H / P, kValueThreads)));
  if (bf16)
    hipLaunchKernelGGL(k_value_rows<BF16>, grid, dim3(kValueThreads), 0, st, static_cast<const uint16_t*>(hidden),
                       ld_hidden, static_cast<const uint16_t*>(w_v), v, ret, mask, T, H, n_ptr,
                       static_cast<uint16_t*>(dhidden_v), part_loss, part_dw);
  else
    hipLaunchKernelGGL(k_value_rows<F32>, grid, dim3(kValueThreads), 0, st, static_cast<const float*>(hidden),
                       ld_hidden, static_cast<const float*>(w_v), v, ret, mask, T, H, n_ptr,
                       static_cast<float*>(dhidden_v), part_loss, part_dw);
  hipLaunchKernelGGL(k_value_final, dim3(static_cast<unsigned>(ceil_div(H, 64))), dim3(kValueThreads), 0,
                     st, part_dw, part_loss, L.row_blocks, H, n_ptr, loss_v, dw_v);
  return hipGetLastError();
}

}  // namespace sao
