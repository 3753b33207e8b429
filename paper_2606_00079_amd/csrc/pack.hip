// Step 5: pack every spectral unit at its assigned width as bit planes with
// fp16 (scale, min) per group, and the inverse (dequantize) for checking.
//
// One wave per unit.  Word w of the row holds entries 64 w .. 64 w + 63, one
// per lane, so the plane-t word of w is the wave ballot of bit t of the lane
// codes.  Words are gathered in LDS and written out contiguously.  Codes
// follow the fp64 quotient rule of the quantizer (decided in fp32 where that
// provably gives the same integer), so they match an fp64 reference bit for
// bit given the same fp32 row.
#include <algorithm>

#include "bitsmoe.h"
#include "common.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

template <int G>
__global__ __launch_bounds__(64) void pack_kernel(const float* __restrict__ C, int64_t units,
                                                  int64_t d, const uint8_t* __restrict__ bits,
                                                  const int64_t* __restrict__ off,
                                                  int64_t total_words,
                                                  uint64_t* __restrict__ codes,
                                                  uint32_t* __restrict__ params) {
  extern __shared__ uint64_t smem[];  // [8 * nw] plane words, then [d/G] params
  constexpr int WPB = G >= 64 ? G / 64 : 1;  // words per group batch
  constexpr int RED = G >= 64 ? 64 : G;      // lanes sharing a group within a word
  const int lane = threadIdx.x;
  const int64_t u = blockIdx.x;
  if (u >= units) return;
  const int b = bits[u];
  const int64_t nw = d / 64;
  const int64_t o0 = off[u], o1 = off[u + 1];
  if (b < 1 || b > BITSMOE_MAX_BITS || o1 - o0 != b * nw || o0 < 0 || o1 > total_words) return;
  uint64_t* wbuf = smem;
  uint32_t* pbuf = reinterpret_cast<uint32_t*>(smem + 8 * nw);
  const double qmax = static_cast<double>((1 << b) - 1);
  const float qmaxf = static_cast<float>((1 << b) - 1);
  const float* crow = C + u * d;
  // words are processed in segments of kSegWords: every load of a segment is
  // issued before any of its values is used
  constexpr int kSegWords = 32;
  static_assert(kSegWords % WPB == 0, "segments hold whole groups");
  for (int64_t s0 = 0; s0 < nw; s0 += kSegWords) {
    float cv[kSegWords];
#pragma unroll
    for (int i = 0; i < kSegWords; ++i) cv[i] = (s0 + i < nw) ? crow[64 * (s0 + i) + lane] : 0.0f;
#pragma unroll
    for (int g0 = 0; g0 < kSegWords; g0 += WPB) {
      const int64_t w0 = s0 + g0;
      if (w0 >= nw) break;
      float mn = cv[g0], mx = cv[g0];
#pragma unroll
      for (int i = 1; i < WPB; ++i) {
        mn = fminf(mn, cv[g0 + i]);
        mx = fmaxf(mx, cv[g0 + i]);
      }
#pragma unroll
      for (int o = RED / 2; o > 0; o >>= 1) {
        mn = fminf(mn, __shfl_xor(mn, o, 64));
        mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      }
      const uint16_t m16 = f32_to_f16_bits(mn);
      const uint16_t s16 = f32_to_f16_bits((mx - mn) / qmaxf);
      const float mf = f16_bits_to_f32(m16);
      const float sf = f16_bits_to_f32(s16);
      // hardware reciprocal (<= 1 ulp): the quotient stays within 6.1e-5 of
      // the fp64 one for codes up to 255, inside the 1e-4 fallback margin
      const float inv = sf > 0.0f ? __builtin_amdgcn_rcpf(sf) : 0.0f;
      // codes from the fp32 quotient: it rounds the same way as the fp64 one
      // unless it lies within 1e-4 of a rounding boundary, and those (rare)
      // lanes decide in fp64
      int q[WPB];
      bool near = false;
#pragma unroll
      for (int i = 0; i < WPB; ++i) {
        const float t = (cv[g0 + i] - mf) * inv;
        const float r = rintf(t);
        near |= fabsf(t - r) > 0.4999f;
        q[i] = static_cast<int>(__builtin_amdgcn_fmed3f(r, 0.0f, qmaxf));
      }
      if (near && sf > 0.0f) {
        const double md = static_cast<double>(mf), sd = static_cast<double>(sf);
#pragma unroll
        for (int i = 0; i < WPB; ++i) {
          const double t = (static_cast<double>(cv[g0 + i]) - md) / sd;
          q[i] = static_cast<int>(fmin(fmax(rint(t), 0.0), qmax));
        }
      }
#pragma unroll
      for (int i = 0; i < WPB; ++i) {
        for (int t = 0; t < b; ++t) {
          const uint64_t word = __ballot((q[i] >> t) & 1);
          if (lane == 0) wbuf[t * nw + w0 + i] = word;
        }
      }
      if ((lane % RED) == 0) {
        const int64_t g = (64 * w0 + lane) / G;
        pbuf[g] = static_cast<uint32_t>(s16) | (static_cast<uint32_t>(m16) << 16);
      }
    }
  }
  __syncthreads();
  for (int64_t i = lane; i < b * nw; i += 64) codes[o0 + i] = wbuf[i];
  const int64_t ng = d / G;
  for (int64_t g = lane; g < ng; g += 64) params[u * ng + g] = pbuf[g];
}

__global__ __launch_bounds__(64) void unpack_kernel(const uint64_t* __restrict__ codes,
                                                    const uint32_t* __restrict__ params,
                                                    const uint8_t* __restrict__ bits,
                                                    const int64_t* __restrict__ off,
                                                    int64_t total_words, int64_t units, int64_t d,
                                                    int G, float* __restrict__ out) {
  const int lane = threadIdx.x;
  const int64_t u = blockIdx.x;
  if (u >= units) return;
  const int b = bits[u];
  const int64_t nw = d / 64;
  const int64_t o0 = off[u], o1 = off[u + 1];
  if (b < 1 || b > BITSMOE_MAX_BITS || o1 - o0 != b * nw || o0 < 0 || o1 > total_words) return;
  const int64_t ng = d / G;
  for (int64_t w = 0; w < nw; ++w) {
    uint32_t q = 0;
    for (int t = 0; t < b; ++t) q |= static_cast<uint32_t>((codes[o0 + t * nw + w] >> lane) & 1u) << t;
    const int64_t k = 64 * w + lane;
    const uint32_t pr = params[u * ng + k / G];
    const float s = f16_bits_to_f32(static_cast<uint16_t>(pr & 0xffffu));
    const float m = f16_bits_to_f32(static_cast<uint16_t>(pr >> 16));
    out[u * d + k] = fmaf(static_cast<float>(q), s, m);
  }
}

bitsmoe_status check_pack_args(int64_t units, int64_t d, int group) {
  if (units <= 0 || d <= 0) return fail(BITSMOE_ERR_ARG, "pack: non-positive size");
  if (!(group == 32 || group == 64 || group == 128 || group == 256))
    return fail(BITSMOE_ERR_SHAPE, "pack: group must be 32, 64, 128 or 256");
  if (d % 64 != 0 || d % group != 0)
    return fail(BITSMOE_ERR_SHAPE, "pack: d must be a multiple of 64 and of the group");
  if (units > INT32_MAX) return fail(BITSMOE_ERR_SHAPE, "pack: too many units");
  return BITSMOE_OK;
}

}  // namespace
}  // namespace bitsmoe

using namespace bitsmoe;

extern "C" bitsmoe_status bitsmoe_pack(const float* C_dev, int64_t units, int64_t d, int group,
                                       const uint8_t* bits_dev, const int64_t* word_offsets_dev,
                                       int64_t total_words, uint64_t* codes_dev,
                                       uint16_t* params_dev, void* stream) {
  if (!C_dev || !bits_dev || !word_offsets_dev || !codes_dev || !params_dev)
    return fail(BITSMOE_ERR_ARG, "pack: null pointer");
  if (!aligned16({C_dev, bits_dev, word_offsets_dev, codes_dev, params_dev}))
    return fail(BITSMOE_ERR_ARG, "pack: device pointers must be 16-byte aligned");
  bitsmoe_status st = check_pack_args(units, d, group);
  if (st != BITSMOE_OK) return st;
  if (total_words < 0) return fail(BITSMOE_ERR_ARG, "pack: negative total_words");
  const size_t lds = static_cast<size_t>(8 * (d / 64)) * 8 + static_cast<size_t>(d / group) * 4;
  if (lds > 160 * 1024) return fail(BITSMOE_ERR_SHAPE, "pack: row too long");
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint32_t* pr = reinterpret_cast<uint32_t*>(params_dev);
  dim3 grid(static_cast<unsigned>(units));
  KernelTimer timer("pack", stream);
  switch (group) {
    case 32:
      hipLaunchKernelGGL(pack_kernel<32>, grid, dim3(64), lds, s, C_dev, units, d, bits_dev,
                         word_offsets_dev, total_words, codes_dev, pr);
      break;
    case 64:
      hipLaunchKernelGGL(pack_kernel<64>, grid, dim3(64), lds, s, C_dev, units, d, bits_dev,
                         word_offsets_dev, total_words, codes_dev, pr);
      break;
    case 128:
      hipLaunchKernelGGL(pack_kernel<128>, grid, dim3(64), lds, s, C_dev, units, d, bits_dev,
                         word_offsets_dev, total_words, codes_dev, pr);
      break;
    default:
      hipLaunchKernelGGL(pack_kernel<256>, grid, dim3(64), lds, s, C_dev, units, d, bits_dev,
                         word_offsets_dev, total_words, codes_dev, pr);
      break;
  }
  BITSMOE_LAUNCH_CHECK("pack: launch");
  return ok();
}

extern "C" bitsmoe_status bitsmoe_unpack(const uint64_t* codes_dev, const uint16_t* params_dev,
                                         const uint8_t* bits_dev, const int64_t* word_offsets_dev,
                                         int64_t total_words, int64_t units, int64_t d, int group,
                                         float* Chat_dev, void* stream) {
  if (!codes_dev || !params_dev || !bits_dev || !word_offsets_dev || !Chat_dev)
    return fail(BITSMOE_ERR_ARG, "unpack: null pointer");
  if (!aligned16({codes_dev, params_dev, bits_dev, word_offsets_dev, Chat_dev}))
    return fail(BITSMOE_ERR_ARG, "unpack: device pointers must be 16-byte aligned");
  bitsmoe_status st = check_pack_args(units, d, group);
  if (st != BITSMOE_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(unpack_kernel, dim3(static_cast<unsigned>(units)), dim3(64), 0, s, codes_dev,
                     reinterpret_cast<const uint32_t*>(params_dev), bits_dev, word_offsets_dev,
                     total_words, units, d, group, Chat_dev);
  BITSMOE_LAUNCH_CHECK("unpack: launch");
  return ok();
}
