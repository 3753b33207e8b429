// Step 5: pack every spectral unit at its assigned width as bit planes with
// fp16 (scale, min) per group, and the inverse (dequantize) for checking.
//
// One wave per unit, four units per workgroup.  Lane l holds entries
// [512 c + 8 l, 512 c + 8 l + 8) of chunk c (a group of G entries spans G/8
// consecutive lanes).  For bit plane t the lane's eight code bits form one
// byte: bit i of it is bit t of entry 8 l + i, which is exactly byte l of the
// plane's 64-bit words 8 c .. 8 c + 7 (word w holds entries 64 w .. 64 w + 63,
// bit j = entry 64 w + j, little-endian), so a plane of a chunk is one
// coalesced 64-byte store.  A row whose length is an odd multiple of 256 ends
// with a 256-entry chunk at 4 entries per lane, each pair of lanes forming
// one byte per plane.  The loads of chunk c + 1 are issued before chunk c is
// packed.  Codes follow the fp64 quotient rule of the quantizer (decided
// in fp32 where that provably gives the same integer), so they match an fp64
// reference bit for bit given the same fp32 row.
#include <algorithm>

#include "bitsmoe.h"
#include "common.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

// Widths a unit may be packed at: codes of 1..8 bits, 16 (fp16 row), 0 (evicted).
__host__ __device__ __forceinline__ bool width_ok(int b) {
  return b == 0 || b == 16 || (b >= 1 && b <= BITSMOE_MAX_BITS);
}

// The bit planes of up to eight codes (each below 256): byte t of the result
// holds bit t of code i in its bit i.  The codes are the rows of an 8 x 8
// bit matrix (code i in byte i of one 64-bit word) and the planes its
// columns, so three rounds of masked swaps (bits one, two and four places
// off the diagonal) transpose it: a few dozen instructions for all eight
// planes instead of three per bit.
template <int N>
__device__ __forceinline__ uint64_t bit_planes(const uint32_t (&q)[N]) {
  static_assert(N <= 8, "eight codes per word");
  uint64_t x = 0;
#pragma unroll
  for (int i = 0; i < N; ++i) x |= static_cast<uint64_t>(q[i]) << (8 * i);
  uint64_t t = (x ^ (x >> 7)) & 0x00AA00AA00AA00AAull;
  x ^= t ^ (t << 7);
  t = (x ^ (x >> 14)) & 0x0000CCCC0000CCCCull;
  x ^= t ^ (t << 14);
  t = (x ^ (x >> 28)) & 0x00000000F0F0F0F0ull;
  x ^= t ^ (t << 28);
  return x;
}

template <int G>
__global__ __launch_bounds__(256) void pack_kernel(const float* __restrict__ C, int64_t units,
                                                   int64_t d, const uint8_t* __restrict__ bits,
                                                   const int64_t* __restrict__ off,
                                                   int64_t total_words,
                                                   uint64_t* __restrict__ codes,
                                                   uint32_t* __restrict__ params) {
  constexpr int GL = G / 8;  // lanes per group
  const int lane = threadIdx.x & 63;
  const int64_t u = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (u >= units) return;  // whole wave exits together
  const int b = bits[u];
  const int64_t nw = d / 64;
  const int64_t o0 = off[u], o1 = off[u + 1];
  if (!width_ok(b) || o1 - o0 != b * nw || o0 < 0 || o1 > total_words) return;
  const float* crow = C + u * d;
  uint32_t* uparams = params + u * (d / G);
  if (b == 0 || b == 16) {
    // eviction stores nothing; width 16 stores the row in fp16, entry k at
    // bits 16 (k % 4) of word k / 4; neither has group parameters
    for (int64_t g = lane; g < d / G; g += 64) uparams[g] = 0u;
    if (b == 16) {
      uint2* w = reinterpret_cast<uint2*>(codes + o0);  // 8-byte aligned words
      for (int64_t k = 4 * lane; k < d; k += 256) {
        const float4 v = *reinterpret_cast<const float4*>(crow + k);
        uint2 h;
        h.x = static_cast<uint32_t>(f32_to_f16_bits(v.x)) | (static_cast<uint32_t>(f32_to_f16_bits(v.y)) << 16);
        h.y = static_cast<uint32_t>(f32_to_f16_bits(v.z)) | (static_cast<uint32_t>(f32_to_f16_bits(v.w)) << 16);
        w[k / 4] = h;
      }
    }
    return;
  }
  const double qmax = static_cast<double>((1 << b) - 1);
  const float qmaxf = static_cast<float>((1 << b) - 1);
  const float rq = 1.0f / qmaxf;
  const float near_at = 0.5f - ldexpf(1.0f, b - 21);  // the fp64 fallback's trigger
  uint8_t* ubytes = reinterpret_cast<uint8_t*>(codes + o0);  // plane t at byte t * d / 8
  // A row whose length is an odd multiple of 256 ends with a chunk of 256
  // entries at 4 per lane (two lanes' nibbles make a byte) instead of a
  // half-empty 512-entry chunk.
  const bool tail4 = d % 512 == 256;
  const int64_t d8 = tail4 ? d - 256 : d;  // the entries of 8-per-lane chunks

  // lane's EPL entries of the chunk at k0 (zeros at or past lim)
  auto load = [&]<int EPL>(int64_t k0, int64_t lim, float (&c)[EPL]) {
    const int64_t k = k0 + EPL * lane;
    if (k < lim) {
#pragma unroll
      for (int i = 0; i < EPL; i += 4) {
        const float4 v = *reinterpret_cast<const float4*>(crow + k + i);
        c[i] = v.x; c[i + 1] = v.y; c[i + 2] = v.z; c[i + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < EPL; ++i) c[i] = 0.0f;
    }
  };
  // codes, group parameters and plane bytes of one chunk
  auto chunk = [&]<int EPL>(int64_t k0, int64_t lim, const float (&c)[EPL]) {
    constexpr int GLE = G / EPL;  // lanes per group
    const int64_t k = k0 + EPL * lane;
    float mn = c[0], mx = c[0];
#pragma unroll
    for (int i = 1; i < EPL; ++i) {
      mn = fminf(mn, c[i]);
      mx = fmaxf(mx, c[i]);
    }
    block_minmax(mn, mx, GLE);
    // d is a multiple of G, so a group is either wholly inside the row or
    // wholly past its end (a 4-entry chunk is always whole)
    if (EPL == 8 && k >= lim) return;
    const uint16_t m16 = f32_to_f16_bits(mn);
    // opaque(): fp16 rounding of the fp32 quotient, not fused into its fma
    const uint16_t s16 = f32_to_f16_bits(opaque(div_qmax(mx - mn, qmaxf, rq)));
    const float mf = f16_bits_to_f32(m16);
    const float sf = f16_bits_to_f32(s16);
    // hardware reciprocal (<= 1 ulp): the fp32 quotient below is within
    // 2^-22 |t| of the fp64 one, and only |t| < 2^b decides a code (further
    // out it is clamped), so it rounds the same way as the fp64 quotient
    // unless it lies within 2^(b-21) of a rounding boundary; those (rare)
    // lanes decide in fp64
    const float inv = sf > 0.0f ? __builtin_amdgcn_rcpf(sf) : 0.0f;
    uint32_t q[EPL];
    bool near = false;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const float t = (c[i] - mf) * inv;
      const float r = rintf(t);
      near |= fabsf(t - r) > near_at;
      q[i] = static_cast<uint32_t>(__builtin_amdgcn_fmed3f(r, 0.0f, qmaxf));
    }
    if (near && sf > 0.0f) {
      // opaque(): the fp64 forms are made inside this branch
      const double md = static_cast<double>(opaque(mf)), sd = static_cast<double>(sf);
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const double t = (static_cast<double>(opaque(c[i])) - md) / sd;
        q[i] = static_cast<uint32_t>(fmin(fmax(rint(t), 0.0), qmax));
      }
    }
    if ((lane % GLE) == 0)
      uparams[k / G] = static_cast<uint32_t>(s16) | (static_cast<uint32_t>(m16) << 16);
    const uint64_t planes = bit_planes(q);
    for (int t = 0; t < b; ++t) {
      const uint32_t bb = static_cast<uint32_t>(planes >> (8 * t)) & 0xFFu;
      if constexpr (EPL == 8) {
        ubytes[t * (d / 8) + k / 8] = static_cast<uint8_t>(bb);
      } else {
        // the odd lane's nibble (entries 4 l + 4 .. 4 l + 7) is the high half
        // of the even lane's byte: lane ^ 1 by a DPP quad permutation
        const uint32_t hi = static_cast<uint32_t>(
            __builtin_amdgcn_mov_dpp(static_cast<int>(bb), 0xB1, 0xF, 0xF, false));
        if ((lane & 1) == 0) ubytes[t * (d / 8) + k / 8] = static_cast<uint8_t>(bb | (hi << 4));
      }
    }
  };
  // the loads of chunk c + 1 are issued before chunk c is packed
  float cur[8], nxt[8];
  load.template operator()<8>(0, d8, cur);
  for (int64_t k0 = 0; k0 < d8; k0 += 512) {
    if (k0 + 512 < d8) load.template operator()<8>(k0 + 512, d8, nxt);
    chunk.template operator()<8>(k0, d8, cur);
#pragma unroll
    for (int i = 0; i < 8; ++i) cur[i] = nxt[i];
  }
  if (tail4) {
    float t[4];
    load.template operator()<4>(d8, d, t);
    chunk.template operator()<4>(d8, d, t);
  }
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
  if (!width_ok(b) || o1 - o0 != b * nw || o0 < 0 || o1 > total_words) return;
  if (b == 0 || b == 16) {
    const uint16_t* h = reinterpret_cast<const uint16_t*>(codes + o0);
    for (int64_t k = lane; k < d; k += 64) out[u * d + k] = b == 0 ? 0.0f : f16_bits_to_f32(h[k]);
    return;
  }
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
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint32_t* pr = reinterpret_cast<uint32_t*>(params_dev);
  dim3 grid(static_cast<unsigned>((units + 3) / 4));
  KernelTimer timer("pack", stream);
  switch (group) {
    case 32:
      hipLaunchKernelGGL(pack_kernel<32>, grid, dim3(256), 0, s, C_dev, units, d, bits_dev,
                         word_offsets_dev, total_words, codes_dev, pr);
      break;
    case 64:
      hipLaunchKernelGGL(pack_kernel<64>, grid, dim3(256), 0, s, C_dev, units, d, bits_dev,
                         word_offsets_dev, total_words, codes_dev, pr);
      break;
    case 128:
      hipLaunchKernelGGL(pack_kernel<128>, grid, dim3(256), 0, s, C_dev, units, d, bits_dev,
                         word_offsets_dev, total_words, codes_dev, pr);
      break;
    default:
      hipLaunchKernelGGL(pack_kernel<256>, grid, dim3(256), 0, s, C_dev, units, d, bits_dev,
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
