// Stage 3: serve one projection of an MoE layer from its packed factors.
//
// The paper dequantizes the packed expert-specific factors inside the expert
// kernels (Sec. 4.4).  With the output-space basis an expert is
// W_e ~ U C^_e, so a token x routed to experts e_j with weights g_j gives
//     y = U z,   z = sum_j g_j C^_{e_j} x,
// the shared basis applied once per token whatever the number of routed
// experts.
//   1. decode_z_kernel  one wave per (expert, unit row): the row is decoded
//                       from its bit planes (or fp16 / evicted widths) once
//                       per chunk of the expert's tokens and dotted with
//                       each token's x: zp[i][k] = w_i (c^_{e,k} . x_{tok_i})
//                       for every routing entry i.
//   2. decode_y_kernel  per token: z = sum of its entries' zp (fixed order),
//                       y = U z with the basis rows read coalesced.
#include <algorithm>
#include <cmath>
#include <string>
#include <vector>

#include "bitsmoe.h"
#include "common.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

constexpr int kTok = 8;  // tokens per pass over a unit row

__device__ __forceinline__ bool width_ok(int b) {
  return b == 0 || b == 16 || (b >= 1 && b <= BITSMOE_MAX_BITS);
}

template <int G>
__global__ __launch_bounds__(256) void decode_z_kernel(
    const uint64_t* __restrict__ codes, const uint32_t* __restrict__ params,
    const uint8_t* __restrict__ bits, const int64_t* __restrict__ off, int64_t total_words,
    int64_t r, int64_t d, const float* __restrict__ X, const int64_t* __restrict__ eoff,
    const int32_t* __restrict__ etok, const float* __restrict__ ew, float* __restrict__ zp) {
  const int lane = threadIdx.x & 63;
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);  // unit of the expert
  const int64_t e = blockIdx.y;
  if (k >= r) return;  // whole wave
  const int64_t i0 = eoff[e], i1 = eoff[e + 1];
  if (i0 >= i1) return;
  const int64_t u = e * r + k;
  const int b = bits[u];
  const int64_t nw = d / 64;
  const int64_t o0 = off[u], o1 = off[u + 1];
  // a unit whose width or offsets are inconsistent contributes nothing (as
  // bitsmoe_pack leaves it unwritten)
  const bool valid = width_ok(b) && b != 0 && o1 - o0 == b * nw && o0 >= 0 && o1 <= total_words;
  const uint32_t* pr = params + u * (d / G);
  const uint16_t* h16 = reinterpret_cast<const uint16_t*>(codes + o0);
  for (int64_t c0 = i0; c0 < i1; c0 += kTok) {
    const int nt = static_cast<int>(std::min<int64_t>(kTok, i1 - c0));
    const float* xs[kTok];
#pragma unroll
    for (int t = 0; t < kTok; ++t) xs[t] = X + static_cast<int64_t>(etok[c0 + (t < nt ? t : nt - 1)]) * d;
    float acc[kTok];
#pragma unroll
    for (int t = 0; t < kTok; ++t) acc[t] = 0.0f;
    if (valid) {
      for (int64_t w = 0; w < nw; ++w) {
        const int64_t j = 64 * w + lane;
        float xh;
        if (b == 16) {
          xh = f16_bits_to_f32(h16[j]);
        } else {
          uint32_t q = 0;
          for (int t = 0; t < b; ++t)
            q |= static_cast<uint32_t>((codes[o0 + t * nw + w] >> lane) & 1u) << t;
          const uint32_t p = pr[j / G];
          const float s = f16_bits_to_f32(static_cast<uint16_t>(p & 0xffffu));
          const float m = f16_bits_to_f32(static_cast<uint16_t>(p >> 16));
          xh = fmaf(static_cast<float>(q), s, m);  // the value bitsmoe_unpack returns
        }
#pragma unroll
        for (int t = 0; t < kTok; ++t) acc[t] = fmaf(xh, xs[t][j], acc[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < kTok; ++t) {
      const float v = wave_sum(acc[t]);
      if (t < nt && lane == 0) zp[(c0 + t) * r + k] = ew[c0 + t] * v;
    }
  }
}

// y[b][o] = sum_k Ut[k][o] z_b[k], z_b[k] = sum over token b's routing entries
// (in the order given) of zp[i][k].
__global__ __launch_bounds__(256) void decode_y_kernel(const float* __restrict__ zp,
                                                       const int64_t* __restrict__ pidx, int kmax,
                                                       int64_t r, const float* __restrict__ Ut,
                                                       int64_t d_out, float* __restrict__ Y) {
  extern __shared__ float z[];  // [r]
  const int64_t b = blockIdx.y;
  const int64_t* pb = pidx + b * kmax;
  for (int64_t k = threadIdx.x; k < r; k += 256) {
    float s = 0.0f;
    for (int j = 0; j < kmax; ++j) {
      const int64_t i = pb[j];
      if (i >= 0) s += zp[i * r + k];
    }
    z[k] = s;
  }
  __syncthreads();
  const int64_t o = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (o >= d_out) return;
  float acc = 0.0f;
  for (int64_t k = 0; k < r; ++k) acc = fmaf(Ut[k * d_out + o], z[k], acc);
  Y[b * d_out + o] = acc;
}

}  // namespace
}  // namespace bitsmoe

using namespace bitsmoe;

extern "C" bitsmoe_status bitsmoe_moe_decode(const uint64_t* codes_dev, const uint16_t* params_dev,
                                             const uint8_t* bits_dev,
                                             const int64_t* word_offsets_dev, int64_t total_words,
                                             int64_t E, int64_t r, int64_t d_in, int group,
                                             const float* Ut_dev, int64_t d_out, const float* X_dev,
                                             int64_t B, const int64_t* offsets_host,
                                             const int32_t* tokens_host, const float* weights_host,
                                             float* Y_dev, void* stream) {
  if (!codes_dev || !params_dev || !bits_dev || !word_offsets_dev || !Ut_dev || !X_dev || !Y_dev ||
      !offsets_host || !tokens_host || !weights_host)
    return fail(BITSMOE_ERR_ARG, "moe_decode: null pointer");
  if (!aligned16({codes_dev, params_dev, bits_dev, word_offsets_dev, Ut_dev, X_dev, Y_dev}))
    return fail(BITSMOE_ERR_ARG, "moe_decode: device pointers must be 16-byte aligned");
  if (E <= 0 || r <= 0 || d_in <= 0 || d_out <= 0 || B <= 0 || total_words < 0)
    return fail(BITSMOE_ERR_ARG, "moe_decode: non-positive size");
  if (E > 65535 || B > 65535) return fail(BITSMOE_ERR_SHAPE, "moe_decode: at most 65535 experts and tokens");
  if (!(group == 32 || group == 64 || group == 128 || group == 256))
    return fail(BITSMOE_ERR_SHAPE, "moe_decode: group must be 32, 64, 128 or 256");
  if (d_in % 64 != 0 || d_in % group != 0)
    return fail(BITSMOE_ERR_SHAPE, "moe_decode: d_in must be a multiple of 64 and of the group");
  if (r > 8192) return fail(BITSMOE_ERR_SHAPE, "moe_decode: r above 8192");
  if (offsets_host[0] != 0) return fail(BITSMOE_ERR_ARG, "moe_decode: offsets[0] must be 0");
  for (int64_t e = 0; e < E; ++e)
    if (offsets_host[e + 1] < offsets_host[e])
      return fail(BITSMOE_ERR_ARG, "moe_decode: offsets must not decrease");
  const int64_t nnz = offsets_host[E];
  // routing entries of each token, in the order given (fixed summation order)
  std::vector<int64_t> cnt(static_cast<size_t>(B), 0);
  for (int64_t i = 0; i < nnz; ++i) {
    if (tokens_host[i] < 0 || tokens_host[i] >= B)
      return fail(BITSMOE_ERR_ARG, "moe_decode: token index outside [0, B)");
    if (!std::isfinite(weights_host[i])) return fail(BITSMOE_ERR_ARG, "moe_decode: non-finite weight");
    ++cnt[static_cast<size_t>(tokens_host[i])];
  }
  int64_t kmax = 1;
  for (int64_t c : cnt) kmax = std::max(kmax, c);
  std::vector<int64_t> pidx(static_cast<size_t>(B * kmax), -1);
  std::fill(cnt.begin(), cnt.end(), 0);
  for (int64_t i = 0; i < nnz; ++i) {
    const int64_t b = tokens_host[i];
    pidx[static_cast<size_t>(b * kmax + cnt[static_cast<size_t>(b)]++)] = i;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  bitsmoe_status st;
  // device tables: expert offsets [E+1], tokens [nnz], weights [nnz], token
  // entry lists [B][kmax]; partials zp [nnz][r]
  const size_t tab_bytes = static_cast<size_t>(E + 1) * 8 + static_cast<size_t>(B * kmax) * 8 +
                           static_cast<size_t>(nnz) * 8 + 64;
  char* tab = static_cast<char*>(scratch(kScratchMisc, tab_bytes, stream, &st));
  if (!tab) return st;
  int64_t* eoff_d = reinterpret_cast<int64_t*>(tab);
  int64_t* pidx_d = eoff_d + (E + 1);
  int32_t* tok_d = reinterpret_cast<int32_t*>(pidx_d + B * kmax);
  float* w_d = reinterpret_cast<float*>(tok_d + nnz + (nnz & 1));
  hipError_t he = hipMemcpyAsync(eoff_d, offsets_host, (E + 1) * 8, hipMemcpyHostToDevice, s);
  if (he == hipSuccess)
    he = hipMemcpyAsync(pidx_d, pidx.data(), B * kmax * 8, hipMemcpyHostToDevice, s);
  if (he == hipSuccess && nnz > 0) he = hipMemcpyAsync(tok_d, tokens_host, nnz * 4, hipMemcpyHostToDevice, s);
  if (he == hipSuccess && nnz > 0) he = hipMemcpyAsync(w_d, weights_host, nnz * 4, hipMemcpyHostToDevice, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);  // host tables may go away after return
  if (he != hipSuccess) return device_error("moe_decode: routing table copy", he);
  float* zp = static_cast<float*>(scratch(kScratchPart, std::max<int64_t>(nnz, 1) * r * 4, stream, &st));
  if (!zp) return st;
  const uint32_t* pr = reinterpret_cast<const uint32_t*>(params_dev);
  {
    KernelTimer timer("moe_decode_z", stream);
    dim3 grid(static_cast<unsigned>((r + 3) / 4), static_cast<unsigned>(E));
#define BITSMOE_DEC(GG)                                                                          \
  hipLaunchKernelGGL(decode_z_kernel<GG>, grid, dim3(256), 0, s, codes_dev, pr, bits_dev,       \
                     word_offsets_dev, total_words, r, d_in, X_dev, eoff_d, tok_d, w_d, zp)
    switch (group) {
      case 32: BITSMOE_DEC(32); break;
      case 64: BITSMOE_DEC(64); break;
      case 128: BITSMOE_DEC(128); break;
      default: BITSMOE_DEC(256); break;
    }
#undef BITSMOE_DEC
  }
  BITSMOE_LAUNCH_CHECK("moe_decode: z launch");
  {
    KernelTimer timer("moe_decode_y", stream);
    dim3 grid(static_cast<unsigned>((d_out + 255) / 256), static_cast<unsigned>(B));
    hipLaunchKernelGGL(decode_y_kernel, grid, dim3(256), static_cast<size_t>(r) * 4, s, zp, pidx_d,
                       static_cast<int>(kmax), r, Ut_dev, d_out, Y_dev);
  }
  BITSMOE_LAUNCH_CHECK("moe_decode: y launch");
  return ok();
}
