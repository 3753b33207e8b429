// Step 4: the activation-aware loss table L[u][j] = delta H delta^T.
//
// For unit row c and width b = bits[j], delta = c - Q_b(c) with the group-wise
// asymmetric round-to-nearest quantizer, and the loss is the exact
// output-space term eps^T H eps of App. B.2 (Eq. app_down_exact_metric),
// written for the unnormalized row.  Split as
//     delta H delta^T = sum_k H_kk delta_k^2  +  delta H_off delta^T,
// the diagonal part is summed in fp32 from the fp32 error, and the
// off-diagonal part, a GEMM of the error rows with H_off, runs on the matrix
// cores in fp16 with fp32 accumulation.  Both fp16 operands are scaled by
// exact powers of two into the upper half of the fp16 range: H_off by 2^F
// (from max |H|), the error rows of unit u by 2^E_u (from max |c_u|), so
// that rows of any magnitude keep fp16's 11-bit precision; the partial sums
// are scaled back by 2^-(2 E_u + F).  (bf16 operands, 8-bit precision, leave
// per-entry errors close to 1e-3 on strongly correlated H; fp16 keeps them
// near 1e-4 at the same matrix-core rate.)
//   1. habsmax_kernel, hoff_kernel
//                    H -> scaled fp16 H_off (zero diagonal), fp32 diag(H)
//   2. dgen_kernel   one wave per unit: max |c_u|, group min/max, fake-quant
//                    at every width, scaled fp16 error rows D[u*nb + j][:] and
//                    the diagonal term of each (u, j)
//   3. gemm          acc[i][row] = sum_k H'[i][k] D[row][k] over the k blocks at
//                    and right of i's block (H' = H_off there, doubled right of
//                    the diagonal block: H is symmetric), epilogue
//                    sum_i D[row][i] acc[i][row] per 256-wide i tile
//   4. finalize      L = diagonal term + the unscaled tile partials, in a fixed
//                    order.
#include <algorithm>
#include <cmath>
#include <string>

#include "bitsmoe.h"
#include "common.hpp"
#include "gemm.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

constexpr int SBM = 256;  // i (H row) tile
constexpr int SBN = 256;  // D row tile
constexpr int SKB = 32;   // K step of the loss-table GEMM
constexpr int SSTAGES = 4;  // LDS stages (two K tiles in flight)
using gemm::BK;

constexpr int kAbsMaxBlocks = 256;  // partial maxima of |H_off|
constexpr int kF16Top = 14;         // scaled fp16 operands stay below 2^14

// Exponent e with 0 <= v < 2^e (v finite, >= 0); 0 for v == 0.
__device__ __forceinline__ int exponent_above(float v) {
  int e = 0;
  (void)frexpf(v, &e);  // v = m 2^e, 0.5 <= m < 1
  return v > 0.0f ? e : 0;
}

// Partial maxima of |H_ik| over the whole matrix (a bound for the
// off-diagonal maximum), one per block; d * d is a multiple of 4.
__global__ __launch_bounds__(256) void habsmax_kernel(const float* __restrict__ H, int64_t d,
                                                      float* __restrict__ partial) {
  __shared__ float red[256];
  H += static_cast<int64_t>(blockIdx.y) * d * d;  // one H per blockIdx.y
  partial += static_cast<int64_t>(blockIdx.y) * kAbsMaxBlocks;
  float m = 0.0f;
  const int64_t n4 = d * d / 4;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  // four 16-byte loads in flight per thread
  for (int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; idx < n4;
       idx += 4 * stride) {
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      v[q] = idx + q * stride < n4 ? reinterpret_cast<const float4*>(H)[idx + q * stride]
                                   : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      m = fmaxf(m, fmaxf(fmaxf(fabsf(v[q].x), fabsf(v[q].y)), fmaxf(fabsf(v[q].z), fabsf(v[q].w))));
  }
  red[threadIdx.x] = m;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + o]);
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[blockIdx.x] = red[0];
}

// H -> fp16 H_off * 2^F (zero diagonal) in the K-tiled layout of 256-row
// tiles (rows padded to a multiple of 256 with zeros), and fp32 diag(H).
// H is symmetric and the GEMM reads only the upper block triangle: row tile
// t uses column blocks t (weight 1) and t + 1, ... (weight 2, which stands
// for the mirrored lower blocks); blocks left of the diagonal are never read.
// F = kF16Top - 1 - e(max |H|), so that doubled entries stay below 2^14;
// block 0 also stores F for the finalize step.
__global__ __launch_bounds__(256) void hoff_kernel(const float* __restrict__ H, int64_t d,
                                                   int64_t d_pad, const float* __restrict__ partial,
                                                   uint16_t* __restrict__ Hoff,
                                                   float* __restrict__ hdiag, int* __restrict__ hexp) {
  __shared__ int sF;
  {  // one H per blockIdx.y
    const int64_t z = blockIdx.y;
    H += z * d * d;
    partial += z * kAbsMaxBlocks;
    Hoff += z * d_pad * d;
    hdiag += z * d;
    hexp += z;
  }
  if (threadIdx.x < 64) {  // wave 0 reduces the partial maxima
    float m = 0.0f;
    for (int b = threadIdx.x; b < kAbsMaxBlocks; b += 64) m = fmaxf(m, partial[b]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if (threadIdx.x == 0) {
      sF = kF16Top - 1 - exponent_above(m);
      if (blockIdx.x == 0) *hexp = sF;
    }
  }
  __syncthreads();
  const int F = sF;
  // eight consecutive outputs per thread: one row i, entries k .. k+7 of one
  // K tile and one column block (d is a multiple of 32)
  const int64_t total8 = d_pad * d / 8;
  const int64_t nkt = d / gemm::kTileK;
  constexpr int64_t TB = static_cast<int64_t>(SBM) * gemm::kTileK;  // elements per tiled block
  for (int64_t c = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; c < total8;
       c += static_cast<int64_t>(gridDim.x) * 256) {
    const int64_t idx = 8 * c;
    const int64_t t = idx / TB, w = idx - t * TB;
    const int64_t rt = t / nkt, kt = t - rt * nkt;
    const int64_t i = rt * SBM + w / gemm::kTileK;
    const int64_t k = kt * gemm::kTileK + w % gemm::kTileK;
    uint16_t v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (i < d && k / SBM >= i / SBM) {  // at or right of the diagonal block
      const float4 h0 = *reinterpret_cast<const float4*>(H + i * d + k);
      const float4 h1 = *reinterpret_cast<const float4*>(H + i * d + k + 4);
      const float h[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
      const int e = k / SBM > i / SBM ? F + 1 : F;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (i == k + q)
          hdiag[i] = h[q];
        else
          v[q] = f32_to_f16_bits(ldexpf(h[q], e));
      }
    }
    uint4 pk;
    pk.x = static_cast<uint32_t>(v[0]) | (static_cast<uint32_t>(v[1]) << 16);
    pk.y = static_cast<uint32_t>(v[2]) | (static_cast<uint32_t>(v[3]) << 16);
    pk.z = static_cast<uint32_t>(v[4]) | (static_cast<uint32_t>(v[5]) << 16);
    pk.w = static_cast<uint32_t>(v[6]) | (static_cast<uint32_t>(v[7]) << 16);
    *reinterpret_cast<uint4*>(Hoff + idx) = pk;
  }
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// The candidate widths, with 2^b - 1, its fp32 reciprocal (the host's
// correctly rounded division) and the fp64 fallback's trigger for each, so
// the kernels read them as arguments instead of deriving them per wave.
//
// The trigger: the fp32 quotient t = (c - m16) * rcp(s16) carries a
// relative error below 2^-22 (fp32 subtraction and product, 2^-24 each, and
// the hardware reciprocal's 1 ulp), and only |t| < 2^b matters (further out
// the code is clamped whatever the rounding), so |t - t_fp64| < 2^(b-22).
// Where t is more than twice that from every half-integer it rounds as the
// fp64 quotient does; closer (|t - rint(t)| > 0.5 - 2^(b-21)) fp64 decides.
struct QuantBits {
  int nb;
  int b[BITSMOE_MAX_NBITS];
  float qmax[BITSMOE_MAX_NBITS];
  float rq[BITSMOE_MAX_NBITS];
  float near[BITSMOE_MAX_NBITS];
  void set(int j, int bits) {
    b[j] = bits;
    qmax[j] = static_cast<float>((1 << bits) - 1);
    rq[j] = 1.0f / qmax[j];
    near[j] = 0.5f - std::ldexp(1.0f, bits - 21);
  }
};

// Group-wise fake quantization of one unit per wave.  Lane l covers entries
// [512 c + 8 l, 512 c + 8 l + 8) of chunk c; a group of G entries spans G/8
// consecutive lanes (with a last chunk of 256 entries at 4 per lane, and G/4
// lanes per group, where the row length is an odd multiple of 256).  Codes
// follow the fp64 rule exactly: the fp32 quotient is used unless it lies
// within 2^(b-21) of a rounding boundary (twice its error bound), in which
// case fp64 decides.
// The row is read twice: once for max |c|, once to quantize.  With ROWLDS
// (rows of at most kRowLds entries) the first pass also keeps the row in
// LDS (8 KiB per wave at 2048 entries) and the second reads it from there,
// so C leaves HBM once; otherwise the second read goes to the caches again
// (holding the row in registers instead costs more in occupancy than it
// saves).  Both passes keep several loads in flight.
//
// NORM: only the error norms are wanted (the input-space table
// beta_k ||delta||^2 of the diagonal approximation): no error rows are
// written, H's diagonal is taken as 1, the errors are not rescaled (E = 0),
// and diag[u * nb + j] = w[u % wperiod] * sum delta^2.
constexpr int kRowLds = 2048;  // longest row dgen_kernel<..., ROWLDS> keeps in LDS

template <int NB, bool NORM = false, bool ROWLDS = false>
__global__ __launch_bounds__(256) void dgen_kernel(const float* __restrict__ C, int64_t units,
                                                   int64_t d, int G, QuantBits qb,
                                                   const float* __restrict__ hdiag,
                                                   uint16_t* __restrict__ D,
                                                   float* __restrict__ diag, int* __restrict__ uexp,
                                                   const float* __restrict__ w = nullptr,
                                                   int64_t wperiod = 1, int64_t hd_upe = 0) {
  const int lane = threadIdx.x & 63;
  const int64_t u = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (u >= units) return;  // whole wave exits together
  constexpr int nb = NB;
  float dacc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) dacc[j] = 0.0f;
  const float* crow = C + u * d;
  if (hd_upe > 0) hdiag += (u / hd_upe) * d;  // one H per block of hd_upe units
  // A row kept in LDS whose length is an odd multiple of 256 ends with a
  // chunk of 256 entries, 4 per lane, instead of a half-empty 512-entry one
  // (d = 768: three quarters of the quantizing work of two full chunks).
  const bool tail4 = ROWLDS && d % 512 == 256;
  const int64_t d8 = tail4 ? d - 256 : d;  // the entries of 8-per-lane chunks

  // lane's EPL entries of the chunk at k0 (EPL * 64 entries; zeros at or past lim)
  auto load = [&]<int EPL>(const float* src, int64_t k0, int64_t lim, float (&c)[EPL]) {
    const int64_t k = k0 + EPL * lane;
    if (k < lim) {
#pragma unroll
      for (int i = 0; i < EPL; i += 4) {
        const float4 v = *reinterpret_cast<const float4*>(src + k + i);
        c[i] = v.x; c[i + 1] = v.y; c[i + 2] = v.z; c[i + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < EPL; ++i) c[i] = 0.0f;
    }
  };
  // ROWLDS: this wave's copy of its row
  __shared__ float rowbuf[ROWLDS ? 4 * kRowLds : 1];
  float* const myrow = rowbuf + (ROWLDS ? (threadIdx.x >> 6) * kRowLds : 0);
  auto keep = [&]<int EPL>(int64_t k0, int64_t lim, const float (&c)[EPL]) {
    if constexpr (ROWLDS) {
      const int64_t k = k0 + EPL * lane;
      if (k < lim) {
#pragma unroll
        for (int i = 0; i < EPL; i += 4)
          *reinterpret_cast<float4*>(myrow + k + i) = make_float4(c[i], c[i + 1], c[i + 2], c[i + 3]);
      }
    }
  };
  // the second pass's copy of the lane's entries
  auto reload = [&]<int EPL>(int64_t k0, int64_t lim, float (&c)[EPL]) {
    load.template operator()<EPL>(ROWLDS ? myrow : crow, k0, lim, c);
  };
  auto absmax = []<int EPL>(const float (&c)[EPL]) {
    float m = 0.0f;
#pragma unroll
    for (int i = 0; i < EPL; ++i) m = fmaxf(m, fabsf(c[i]));
    return m;
  };

  // |delta| <= max - min <= 2 max |c| < 2^(e + 1): the error rows are stored
  // as fp16(delta * 2^E) with E = kF16Top - 1 - e.  Every load of a group of
  // chunks (four 8-entry chunks, or what is left of the row) is issued
  // before any is reduced.
  int E = 0;
  if constexpr (!NORM) {
    float amax = 0.0f;
    int64_t ka = 0;
    for (; ka + 4 * 512 <= d8; ka += 4 * 512) {
      float c4[4][8];
#pragma unroll
      for (int x = 0; x < 4; ++x) load.template operator()<8>(crow, ka + 512 * x, d8, c4[x]);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        amax = fmaxf(amax, absmax.template operator()<8>(c4[x]));
        keep.template operator()<8>(ka + 512 * x, d8, c4[x]);
      }
    }
    {
      float c4[4][8], t[4];
#pragma unroll
      for (int x = 0; x < 4; ++x)
        if (ka + 512 * x < d8) load.template operator()<8>(crow, ka + 512 * x, d8, c4[x]);
      if (tail4) load.template operator()<4>(crow, d8, d, t);
#pragma unroll
      for (int x = 0; x < 4; ++x)
        if (ka + 512 * x < d8) {
          amax = fmaxf(amax, absmax.template operator()<8>(c4[x]));
          keep.template operator()<8>(ka + 512 * x, d8, c4[x]);
        }
      if (tail4) {
        amax = fmaxf(amax, absmax.template operator()<4>(t));
        keep.template operator()<4>(d8, d, t);
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
    E = kF16Top - 1 - exponent_above(amax);
    if (lane == 0) uexp[u] = E;
  }

  // quantize one chunk (EPL entries per lane) at every width
  auto chunk = [&]<int EPL>(int64_t k0, int64_t lim, const float (&c)[EPL]) {
    const int64_t k = k0 + EPL * lane;
    const bool active = k < lim;
    float mn = c[0], mx = c[0];
#pragma unroll
    for (int i = 1; i < EPL; ++i) {
      mn = fminf(mn, c[i]);
      mx = fmaxf(mx, c[i]);
    }
    block_minmax(mn, mx, G / EPL);
    if (!active) return;
    float hd[EPL];
    if constexpr (NORM) {
#pragma unroll
      for (int i = 0; i < EPL; ++i) hd[i] = 1.0f;
    } else {
      load.template operator()<EPL>(hdiag, k0, lim, hd);
    }
    const float mf = f16_bits_to_f32(f32_to_f16_bits(mn));
    const float range = mx - mn;
    // c - m16 once per entry, and its image scaled by 2^E (exact)
    float cm[EPL], cms[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      cm[i] = c[i] - mf;
      cms[i] = ldexpf(cm[i], E);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const float qmax = qb.qmax[j];
      // opaque(): the fp16 rounding below must apply to the fp32 quotient,
      // not be fused into its last fma (which would round the exact sum once)
      const float s32 = opaque(div_qmax(range, qmax, qb.rq[j]));
      const float sf = f16_bits_to_f32(f32_to_f16_bits(s32));
      // hardware reciprocal (<= 1 ulp)
      const float inv = sf > 0.0f ? __builtin_amdgcn_rcpf(sf) : 0.0f;
      const float sfs = ldexpf(sf, E);
      // codes from the fp32 quotient (inv = 0 gives q = 0 for a constant
      // group); a quotient within 2^(b-21) of a rounding boundary is decided
      // in fp64 instead, for the whole lane, in one rarely taken branch
      const float near_at = qb.near[j];
      float q[EPL];
      bool near = false;
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const float t = cm[i] * inv;
        const float r = rintf(t);
        near |= fabsf(t - r) > near_at;
        q[i] = __builtin_amdgcn_fmed3f(r, 0.0f, qmax);
      }
      if (near && sf > 0.0f) {
        // The entries are read again (from the LDS copy, or through the
        // caches) rather than kept in registers through every width.  Each
        // entry's operand passes through an empty asm that also takes the
        // previous entry's code: the fp64 work stays inside this branch and
        // runs one entry at a time, so its registers do not add up over the
        // entries (they would set the kernel's register count).
        const float* src = (ROWLDS ? myrow : crow) + k;
        const double md = static_cast<double>(mf);
        const double sd = static_cast<double>(sf);
        float prev = 0.0f;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
          float x = src[i];
          asm volatile("" : "+v"(x) : "v"(prev));
          const double td = (static_cast<double>(x) - md) / sd;
          q[i] = static_cast<float>(fmin(fmax(rint(td), 0.0), static_cast<double>(qmax)));
          prev = q[i];
        }
      }
      // delta * 2^E = (c - m16) 2^E - q s16 2^E; the diagonal term is summed
      // from the scaled error and scaled back once at the end
      float dls[EPL];
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        dls[i] = fmaf(-q[i], sfs, cms[i]);
        dacc[j] = fmaf(hd[i] * dls[i], dls[i], dacc[j]);
      }
      if constexpr (!NORM) {
        // two fp16 per instruction (the fp32 value rounded to nearest even)
        uint32_t pk[EPL / 2];
#pragma unroll
        for (int i = 0; i < EPL; i += 2)
          pk[i / 2] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{dls[i], dls[i + 1]}, f16x2));
        uint16_t* dst = D + gemm::tiled_offset(u * nb + j, k, d, SBN);
        if constexpr (EPL == 8)
          *reinterpret_cast<uint4*>(dst) = make_uint4(pk[0], pk[1], pk[2], pk[3]);
        else
          *reinterpret_cast<uint2*>(dst) = make_uint2(pk[0], pk[1]);
      }
    }
  };
  // the loads of chunk c + 1 are issued before chunk c is quantized
  static_assert(!(NORM && ROWLDS), "the norm-only form has no first pass");
  float cur[8], nxt[8];
  reload.template operator()<8>(0, d8, cur);
  for (int64_t k0 = 0; k0 < d8; k0 += 512) {
    if (k0 + 512 < d8) reload.template operator()<8>(k0 + 512, d8, nxt);
    chunk.template operator()<8>(k0, d8, cur);
#pragma unroll
    for (int i = 0; i < 8; ++i) cur[i] = nxt[i];
  }
  if (tail4) {
    float t[4];
    reload.template operator()<4>(d8, d, t);
    chunk.template operator()<4>(d8, d, t);
  }
  const float wu = NORM ? w[u % wperiod] : 1.0f;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const float v = ldexpf(wave_sum(dacc[j]), -2 * E);
    if (lane == 0) diag[u * nb + j] = NORM ? wu * v : v;
  }
}

// part[row][tm] = sum over this tile's i of D[row][i] * acc[i][row].
//
// The i range of the tile is K tiles 8 tm .. 8 tm + 7 of D (the diagonal
// block), which the K loop visits last, in descending order: the first four
// (the i range of the waves with wm = 0) are the last four tiles staged and
// are still in the B halves of the stage buffers; the other four (wm = 1)
// are loaded again into the A halves, which are free once the loop is done.
// Both use the stage layout (256 rows x 32 entries, swizzled 16-byte
// chunks).  Each lane then reads its D values (one row per column fragment,
// four 8-byte runs per row fragment).  K tiles past the end of the row are
// clamped (their accumulators are exactly zero: H_off's pad rows are zero);
// rows past the end (the padding of the last row tile) are computed and
// never stored.
struct RowDot {
  static constexpr bool kUsesLds = true;  // reads or writes the stage buffers
  const uint16_t* D;
  float* part;
  int64_t R, d;
  int tiles_m;
  template <class F>
  __device__ void operator()(F& f, const gemm::StageLds& lds) const {
    static_assert(SBM == 256 && SBN == 256 && SKB == 32 && SSTAGES >= 4,
                  "layout below assumes 256 x 256 tiles, 32-wide K tiles, four or more stages");
    constexpr int TE = SBN * SKB;  // elements of one staged K tile of D (and of H_off)
    __shared__ float red[2 * SBN];  // cross-wave reduction
    const int lane = opaque(f.lane);
    const int wave = lane >= 0 ? f.wave : 0;  // ties wave to the opaque lane
    const int64_t nkt = d / gemm::kTileK;
    const int64_t kt0 = static_cast<int64_t>(f.tm) * (SBM / SKB);  // first K tile of the block
    const uint16_t* dtile = D + static_cast<int64_t>(f.tn) * SBN * d;  // row tile tn of D
    // reload block K tiles 4..7 (clamped) into A buffers 0..3
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int64_t q = min(kt0 + 4 + x, nkt - 1);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int blk = wave + 4 * i;                 // 1 KiB block: rows 16 blk .. 16 blk + 15
        const int r = 16 * blk + (lane >> 2);
        const int j = gemm::swz<SKB>(r, lane & 3);
        gemm::dma16(dtile + q * TE, static_cast<uint32_t>((r * SKB + 8 * j) * 2),
                    lds.a + x * TE + blk * 512);
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    float s[F::FN];
#pragma unroll
    for (int ni = 0; ni < F::FN; ++ni) {
      // one column fragment at a time: keeps the LDS reads from being hoisted
      // next to all 256 accumulators
      __builtin_amdgcn_sched_barrier(0);
      const int jl = f.wn * F::WN + 32 * ni + (lane & 31);
      float acc = 0.0f;
#pragma unroll
      for (int mi = 0; mi < F::FM; ++mi) {
        const int rq = 4 * f.wm + mi;  // block K tile (uniform per wave)
        // rq < 4: staged as visit n = nk - 1 - rq, still in B buffer n % stages
        const int64_t n = lds.nk - 1 - rq;
        const uint16_t* tb = rq < 4 ? lds.b + static_cast<int>((n < 0 ? 0 : n) % lds.stages) * TE
                                    : lds.a + (rq - 4) * TE;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int k = 8 * g + 4 * (lane >> 5);  // entry within the K tile
          const uint2 v = *reinterpret_cast<const uint2*>(tb + gemm::lds_off<SKB>(jl, k >> 3) + (k & 7));
          const _Float16* h = reinterpret_cast<const _Float16*>(&v);
          acc = fmaf(static_cast<float>(h[0]), f.acc[mi][ni][4 * g + 0], acc);
          acc = fmaf(static_cast<float>(h[1]), f.acc[mi][ni][4 * g + 1], acc);
          acc = fmaf(static_cast<float>(h[2]), f.acc[mi][ni][4 * g + 2], acc);
          acc = fmaf(static_cast<float>(h[3]), f.acc[mi][ni][4 * g + 3], acc);
        }
      }
      s[ni] = acc + __shfl_xor(acc, 32, 64);
    }
    // combine the waves that share these rows (wm = 0, 1)
    if ((lane >> 5) == 0) {
#pragma unroll
      for (int ni = 0; ni < F::FN; ++ni) red[f.wm * SBN + f.wn * F::WN + 32 * ni + lane] = s[ni];
    }
    __syncthreads();
    const int64_t j_base = static_cast<int64_t>(f.tn) * SBN;
    for (int t = threadIdx.x; t < SBN; t += gemm::kThreads) {
      const int64_t row = j_base + t;
      if (row < R) part[row * tiles_m + f.tm] = red[t] + red[SBN + t];
    }
  }
};

// L = diagonal term + (sum of the tile partials, in tile order) * 2^-(2 E_u + F).
// With one H per block of upe units (upe > 0), the H exponent is that H's.
__global__ __launch_bounds__(256) void finalize_kernel(const float* __restrict__ diag,
                                                       const float* __restrict__ part, int64_t R,
                                                       int tiles_m, int nb,
                                                       const int* __restrict__ uexp,
                                                       const int* __restrict__ hexp,
                                                       float* __restrict__ L, int64_t upe = 0) {
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (row >= R) return;
  const float* p = part + row * tiles_m;
  float s = 0.0f;
  for (int t = 0; t < tiles_m; ++t) s += p[t];
  const int64_t u = row / nb;
  const int F = hexp[upe > 0 ? u / upe : 0];
  L[row] = diag[row] + ldexpf(s, -(2 * uexp[u] + F));
}

// Raw rows for the surrogate's activation-aware importance (the eviction
// case of the loss table, delta = c): one wave per unit writes fp16(c 2^E)
// in the K-tiled layout of the loss-table GEMM, the diagonal term
// sum_k H_kk c_k^2, and the fp32 row statistics sum c^2, max |c|, sum |c|.
__global__ __launch_bounds__(256) void rowprep_kernel(const float* __restrict__ C, int64_t units,
                                                      int64_t d, const float* __restrict__ hdiag,
                                                      uint16_t* __restrict__ D,
                                                      float* __restrict__ diag,
                                                      int* __restrict__ uexp,
                                                      float* __restrict__ rstats) {
  const int lane = threadIdx.x & 63;
  const int64_t u = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (u >= units) return;  // whole wave exits together
  const float* crow = C + u * d;
  auto load8 = [&](int64_t k0, float (&c)[8]) {
    const int64_t k = k0 + 8 * lane;
    if (k < d) {
      const float4 v0 = *reinterpret_cast<const float4*>(crow + k);
      const float4 v1 = *reinterpret_cast<const float4*>(crow + k + 4);
      c[0] = v0.x; c[1] = v0.y; c[2] = v0.z; c[3] = v0.w;
      c[4] = v1.x; c[5] = v1.y; c[6] = v1.z; c[7] = v1.w;
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) c[i] = 0.0f;
    }
  };
  // pass 1: max |c|, sum c^2, sum |c|, four chunks' loads in flight
  float amax = 0.0f, s2 = 0.0f, s1 = 0.0f;
  auto acc8 = [&](const float (&c)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      amax = fmaxf(amax, fabsf(c[i]));
      s2 = fmaf(c[i], c[i], s2);
      s1 += fabsf(c[i]);
    }
  };
  int64_t ka = 0;
  for (; ka + 4 * 512 <= d; ka += 4 * 512) {
    float c4[4][8];
#pragma unroll
    for (int x = 0; x < 4; ++x) load8(ka + 512 * x, c4[x]);
#pragma unroll
    for (int x = 0; x < 4; ++x) acc8(c4[x]);
  }
  for (; ka < d; ka += 512) {
    float cc[8];
    load8(ka, cc);
    acc8(cc);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  s2 = wave_sum(s2);
  s1 = wave_sum(s1);
  // |c| < 2^e: the rows are stored as fp16(c 2^E), E = kF16Top - 1 - e
  const int E = kF16Top - 1 - exponent_above(amax);
  // pass 2: scaled fp16 rows and the diagonal term
  float dacc = 0.0f;
  float cur[8], nxt[8];
  load8(0, cur);
  for (int64_t k0 = 0; k0 < d; k0 += 512) {
    if (k0 + 512 < d) load8(k0 + 512, nxt);
    const int64_t k = k0 + 8 * lane;
    if (k < d) {
      const float4 h0 = *reinterpret_cast<const float4*>(hdiag + k);
      const float4 h1 = *reinterpret_cast<const float4*>(hdiag + k + 4);
      const float hd[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
      uint16_t out[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float cs = ldexpf(cur[i], E);
        out[i] = f32_to_f16_bits(cs);
        dacc = fmaf(hd[i] * cs, cs, dacc);
      }
      uint4 pk;
      pk.x = static_cast<uint32_t>(out[0]) | (static_cast<uint32_t>(out[1]) << 16);
      pk.y = static_cast<uint32_t>(out[2]) | (static_cast<uint32_t>(out[3]) << 16);
      pk.z = static_cast<uint32_t>(out[4]) | (static_cast<uint32_t>(out[5]) << 16);
      pk.w = static_cast<uint32_t>(out[6]) | (static_cast<uint32_t>(out[7]) << 16);
      *reinterpret_cast<uint4*>(D + gemm::tiled_offset(u, k, d, SBN)) = pk;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) cur[i] = nxt[i];
  }
  dacc = ldexpf(wave_sum(dacc), -2 * E);
  if (lane == 0) {
    uexp[u] = E;
    diag[u] = dacc;
    rstats[3 * u + 0] = s2;
    rstats[3 * u + 1] = amax;
    rstats[3 * u + 2] = s1;
  }
}

// Low-bit distortion coefficients of the surrogate (widths 2, 3, 4).
struct Kappa {
  double k[3];
};

// The surrogate table of one unit (App. B.3-B.4): alpha^2 = sum c^2,
// beta = c H c^T / alpha^2, rho = max |c| / alpha, cos theta =
// sum |c| / (alpha sqrt(d)); L[u][j] = alpha^2 beta^gamma E(width j) over the
// widths 0, 1, 2, 3, 4, 6, 8, 16.  A zero row costs 0 everywhere.
__global__ __launch_bounds__(256) void surrogate_finalize_kernel(
    const float* __restrict__ diag, const float* __restrict__ part, int64_t units, int tiles_m,
    const int* __restrict__ uexp, const int* __restrict__ hexp, const float* __restrict__ rstats,
    int64_t d, double gamma, Kappa kap, float* __restrict__ L, float* __restrict__ stats_out) {
  const int64_t u = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (u >= units) return;
  const float* p = part + u * tiles_m;
  float s = 0.0f;
  for (int t = 0; t < tiles_m; ++t) s += p[t];
  const double q = static_cast<double>(diag[u] + ldexpf(s, -(2 * uexp[u] + *hexp)));  // c H c^T
  const double a2 = static_cast<double>(rstats[3 * u + 0]);
  double beta = 0.0, rho = 0.0, cs = 0.0, w = 0.0;
  if (a2 > 0.0) {
    const double alpha = sqrt(a2);
    beta = q / a2;
    rho = static_cast<double>(rstats[3 * u + 1]) / alpha;
    // ||p||_1 <= sqrt(d) (Cauchy-Schwarz); rows of equal magnitudes attain it
    cs = fmin(static_cast<double>(rstats[3 * u + 2]) / (alpha * sqrt(static_cast<double>(d))), 1.0);
    w = a2 * pow(fmax(beta, 0.0), gamma);
  }
  const double eta = static_cast<double>(d) * rho * rho / 3.0;
  float* row = L + u * BITSMOE_SURROGATE_NWIDTHS;
  row[0] = static_cast<float>(w);                       // b = 0: eviction, E = 1
  row[1] = static_cast<float>(w * (1.0 - cs) * (1.0 + cs));  // b = 1: sin^2 theta
  row[2] = static_cast<float>(w * kap.k[0]);            // b = 2
  row[3] = static_cast<float>(w * kap.k[1]);            // b = 3
  row[4] = static_cast<float>(w * kap.k[2]);            // b = 4
  row[5] = static_cast<float>(w * eta * ldexp(1.0, -12));  // b = 6: eta 4^-6
  row[6] = static_cast<float>(w * eta * ldexp(1.0, -16));  // b = 8
  row[7] = static_cast<float>(w * eta * ldexp(1.0, -32));  // b = 16
  if (stats_out) {
    stats_out[4 * u + 0] = static_cast<float>(a2);
    stats_out[4 * u + 1] = static_cast<float>(beta);
    stats_out[4 * u + 2] = static_cast<float>(rho);
    stats_out[4 * u + 3] = static_cast<float>(cs);
  }
}

// q[row] = c H c^T for the raw rows prepared by rowprep_kernel.
__global__ __launch_bounds__(256) void quadform_finalize_kernel(const float* __restrict__ diag,
                                                                const float* __restrict__ part,
                                                                int64_t rows, int tiles_m,
                                                                const int* __restrict__ uexp,
                                                                const int* __restrict__ hexp,
                                                                float* __restrict__ q) {
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (row >= rows) return;
  const float* p = part + row * tiles_m;
  float s = 0.0f;
  for (int t = 0; t < tiles_m; ++t) s += p[t];
  q[row] = diag[row] + ldexpf(s, -(2 * uexp[row] + *hexp));
}

// Scratch and launch shape of one loss-table evaluation over R rows of D
// (error rows for the score, raw rows for the surrogate) against H.
struct LossTable {
  int64_t d, R, units;
  int64_t nh;        // number of H matrices (one per block of units / nh units)
  int tiles_m;
  int64_t tiles_n, d_pad, R_pad;
  uint16_t* Hoff;
  uint16_t* D;
  float* hdiag;  // [d]
  float* diag;   // [R]
  int* uexp;     // [units]
  float* hpart;  // [kAbsMaxBlocks]
  int* hexp;     // [nh]
  float* rstats; // [3 units] (surrogate only)
  float* part;   // [R][tiles_m]
};

bitsmoe_status loss_table_setup(int64_t d, int64_t R, int64_t units, bool row_stats, void* stream,
                                const char* who, LossTable* t, int64_t nh = 1) {
  t->d = d;
  t->R = R;
  t->units = units;
  t->nh = nh;
  t->tiles_m = static_cast<int>((d + SBM - 1) / SBM);
  t->tiles_n = (R + SBN - 1) / SBN;
  if (gemm::paired_workgroups(t->tiles_m, t->tiles_n) > INT32_MAX || (R + 255) / 256 > INT32_MAX)
    return fail(BITSMOE_ERR_SHAPE, std::string(who) + ": too many units");
  // H_off and D are K-tiled with 256-row tiles, rows padded to whole tiles
  t->d_pad = t->tiles_m * static_cast<int64_t>(SBM);
  t->R_pad = t->tiles_n * static_cast<int64_t>(SBN);
  bitsmoe_status st;
  t->Hoff = static_cast<uint16_t*>(scratch(kScratchA, nh * t->d_pad * d * 2, stream, &st));
  if (!t->Hoff) return st;
  // small tables: diag(H) [nh][d], diagonal terms [R], unit exponents
  // [units], partial maxima of |H_off| [nh][kAbsMaxBlocks], the H_off
  // exponents [nh], row statistics [3 units]
  const int64_t small_words =
      nh * d + R + units + nh * kAbsMaxBlocks + nh + (row_stats ? 3 * units : 0);
  float* small = static_cast<float*>(scratch(kScratchMisc, small_words * sizeof(float), stream, &st));
  if (!small) return st;
  t->hdiag = small;
  t->diag = t->hdiag + nh * d;
  t->uexp = reinterpret_cast<int*>(t->diag + R);
  t->hpart = reinterpret_cast<float*>(t->uexp + units);
  t->hexp = reinterpret_cast<int*>(t->hpart + nh * kAbsMaxBlocks);
  t->rstats = row_stats ? reinterpret_cast<float*>(t->hexp + nh) : nullptr;
  t->D = static_cast<uint16_t*>(scratch(kScratchD, t->R_pad * d * 2, stream, &st));
  if (!t->D) return st;
  t->part = static_cast<float*>(scratch(kScratchPart, R * t->tiles_m * sizeof(float), stream, &st));
  if (!t->part) return st;
  return BITSMOE_OK;
}

// H -> scaled fp16 H_off and diag(H).
bitsmoe_status loss_table_hoff(const float* H_dev, const LossTable& t, hipStream_t s, const char* who) {
  const unsigned nh = static_cast<unsigned>(t.nh);
  hipLaunchKernelGGL(habsmax_kernel, dim3(kAbsMaxBlocks, nh), dim3(256), 0, s, H_dev, t.d, t.hpart);
  BITSMOE_LAUNCH_CHECK(who);
  const unsigned hb = static_cast<unsigned>(std::min<int64_t>((t.d_pad * t.d / 8 + 255) / 256, 16384));
  hipLaunchKernelGGL(hoff_kernel, dim3(hb, nh), dim3(256), 0, s, H_dev, t.d, t.d_pad, t.hpart, t.Hoff,
                     t.hdiag, t.hexp);
  BITSMOE_LAUNCH_CHECK(who);
  return BITSMOE_OK;
}

// part[row][tm] = sum over the 256-wide tile tm of H rows of the
// off-diagonal form of row `row` of D (paired upper-triangle schedule).
// With t.nh > 1, column tile tn of D multiplies H number (tn * 256) /
// a_batch_rows (every block of a_batch_rows rows of D belongs to one H).
bitsmoe_status loss_table_gemm(const LossTable& t, void* stream, const char* timer, const char* who,
                               int64_t a_batch_rows = 0) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  gemm::Problem p{};
  static_assert(SKB == gemm::kTileK, "the K-tiled operands need the kernel's K step");
  p.a.pass[0] = t.Hoff;
  p.a.rows = t.d_pad;
  p.a.kstep = static_cast<int64_t>(SBM) * gemm::kTileK;
  p.a.rtile = static_cast<int64_t>(SBM) * t.d;
  p.a.bstride = t.d_pad * t.d;
  p.a_batch_rows = a_batch_rows;
  p.b.pass[0] = t.D;
  p.b.rows = t.R_pad;
  p.b.kstep = static_cast<int64_t>(SBN) * gemm::kTileK;
  p.b.rtile = static_cast<int64_t>(SBN) * t.d;
  p.passes = 1;
  p.segs = 1;
  p.kseg = t.d;
  p.ktiles = t.d / BK;
  p.splits = 1;
  p.tiles_m = t.tiles_m;
  p.tiles_n = static_cast<int>(t.tiles_n);
  p.symmetric = 0;
  // H symmetric: only the upper block triangle of H_off is visited, in the
  // paired schedule, so that every workgroup does the same tiles_m + 1
  // blocks of work
  p.group_n = std::max(1, 32 / gemm::paired_unit_workgroups(t.tiles_m));  // ~one XCD's worth
  RowDot epi{t.D, t.part, t.R, t.d, t.tiles_m};
  dim3 grid(static_cast<unsigned>(gemm::paired_workgroups(t.tiles_m, t.tiles_n)), 1, 1);
  {
    KernelTimer kt(timer, stream);
    hipLaunchKernelGGL((gemm::gemm_nt_kernel<SBM, SBN, SKB, SSTAGES, RowDot, true, false, true>),
                       grid, dim3(gemm::kThreads), 0, s, p, epi);
  }
  BITSMOE_LAUNCH_CHECK(who);
  return BITSMOE_OK;
}

bitsmoe_status check_rows_args(const float* C_dev, const float* H_dev, int64_t units, int64_t d,
                               const char* who) {
  if (!aligned16({C_dev, H_dev}))
    return fail(BITSMOE_ERR_ARG, std::string(who) + ": device pointers must be 16-byte aligned");
  if (units <= 0 || d <= 0) return fail(BITSMOE_ERR_ARG, std::string(who) + ": non-positive size");
  if (d % 64 != 0) return fail(BITSMOE_ERR_SHAPE, std::string(who) + ": d must be a multiple of 64");
  if (d >= (int64_t{1} << 22)) return fail(BITSMOE_ERR_SHAPE, std::string(who) + ": d must be below 2^22");
  return BITSMOE_OK;
}

}  // namespace
}  // namespace bitsmoe

using namespace bitsmoe;

extern "C" bitsmoe_status bitsmoe_score(const float* C_dev, int64_t units, int64_t d,
                                        const float* H_dev, const int* bits_host, int nbits,
                                        int group, float* L_dev, void* stream) {
  if (!C_dev || !H_dev || !bits_host || !L_dev) return fail(BITSMOE_ERR_ARG, "score: null pointer");
  if (!aligned16({L_dev})) return fail(BITSMOE_ERR_ARG, "score: device pointers must be 16-byte aligned");
  bitsmoe_status st = check_rows_args(C_dev, H_dev, units, d, "score");
  if (st != BITSMOE_OK) return st;
  if (nbits < 1 || nbits > BITSMOE_MAX_NBITS) return fail(BITSMOE_ERR_ARG, "score: nbits outside 1..8");
  QuantBits qb{};
  qb.nb = nbits;
  for (int j = 0; j < nbits; ++j) {
    if (bits_host[j] < 1 || bits_host[j] > BITSMOE_MAX_BITS)
      return fail(BITSMOE_ERR_ARG, "score: width outside 1..8");
    if (j > 0 && bits_host[j] <= bits_host[j - 1])
      return fail(BITSMOE_ERR_ARG, "score: widths must be strictly ascending");
    qb.set(j, bits_host[j]);
  }
  if (!(group == 32 || group == 64 || group == 128 || group == 256))
    return fail(BITSMOE_ERR_SHAPE, "score: group must be 32, 64, 128 or 256");
  if (d % group != 0) return fail(BITSMOE_ERR_SHAPE, "score: d must be a multiple of the group");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t R = units * nbits;
  LossTable t;
  st = loss_table_setup(d, R, units, false, stream, "score", &t);
  if (st != BITSMOE_OK) return st;
  st = loss_table_hoff(H_dev, t, s, "score: H_off launch");
  if (st != BITSMOE_OK) return st;
  const unsigned db = static_cast<unsigned>((units + 3) / 4);
  {
  KernelTimer dgen_timer("score_dgen", stream);
  switch (nbits) {
#define BITSMOE_DGEN(NB)                                                                         \
  case NB:                                                                                       \
    if (d <= kRowLds)                                                                            \
      hipLaunchKernelGGL((dgen_kernel<NB, false, true>), dim3(db), dim3(256), 0, s, C_dev, units, \
                         d, group, qb, t.hdiag, t.D, t.diag, t.uexp);                            \
    else                                                                                         \
      hipLaunchKernelGGL((dgen_kernel<NB, false, false>), dim3(db), dim3(256), 0, s, C_dev,      \
                         units, d, group, qb, t.hdiag, t.D, t.diag, t.uexp);                     \
    break;
    BITSMOE_DGEN(1) BITSMOE_DGEN(2) BITSMOE_DGEN(3) BITSMOE_DGEN(4)
    BITSMOE_DGEN(5) BITSMOE_DGEN(6) BITSMOE_DGEN(7) BITSMOE_DGEN(8)
#undef BITSMOE_DGEN
  }
  }
  BITSMOE_LAUNCH_CHECK("score: dgen launch");
  st = loss_table_gemm(t, stream, "score_gemm", "score: gemm launch");
  if (st != BITSMOE_OK) return st;
  hipLaunchKernelGGL(finalize_kernel, dim3(static_cast<unsigned>((R + 255) / 256)), dim3(256), 0, s,
                     t.diag, t.part, R, t.tiles_m, nbits, t.uexp, t.hexp, L_dev);
  BITSMOE_LAUNCH_CHECK("score: finalize launch");
  return ok();
}

extern "C" bitsmoe_status bitsmoe_surrogate(const float* C_dev, int64_t units, int64_t d,
                                            const float* H_dev, double gamma,
                                            const double* kappa_host, float* L_dev,
                                            float* stats_dev, void* stream) {
  if (!C_dev || !H_dev || !kappa_host || !L_dev) return fail(BITSMOE_ERR_ARG, "surrogate: null pointer");
  if (!aligned16({L_dev, stats_dev}))
    return fail(BITSMOE_ERR_ARG, "surrogate: device pointers must be 16-byte aligned");
  bitsmoe_status st = check_rows_args(C_dev, H_dev, units, d, "surrogate");
  if (st != BITSMOE_OK) return st;
  if (!(gamma >= 0.0 && gamma <= 1.0)) return fail(BITSMOE_ERR_ARG, "surrogate: gamma outside [0, 1]");
  Kappa kap{};
  for (int j = 0; j < 3; ++j) {
    if (!(kappa_host[j] >= 0.0) || !std::isfinite(kappa_host[j]))
      return fail(BITSMOE_ERR_ARG, "surrogate: kappa must be finite and non-negative");
    kap.k[j] = kappa_host[j];
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  LossTable t;
  st = loss_table_setup(d, units, units, true, stream, "surrogate", &t);
  if (st != BITSMOE_OK) return st;
  st = loss_table_hoff(H_dev, t, s, "surrogate: H_off launch");
  if (st != BITSMOE_OK) return st;
  {
    KernelTimer rt("surrogate_rows", stream);
    hipLaunchKernelGGL(rowprep_kernel, dim3(static_cast<unsigned>((units + 3) / 4)), dim3(256), 0, s,
                       C_dev, units, d, t.hdiag, t.D, t.diag, t.uexp, t.rstats);
  }
  BITSMOE_LAUNCH_CHECK("surrogate: row launch");
  st = loss_table_gemm(t, stream, "surrogate_gemm", "surrogate: gemm launch");
  if (st != BITSMOE_OK) return st;
  hipLaunchKernelGGL(surrogate_finalize_kernel, dim3(static_cast<unsigned>((units + 255) / 256)),
                     dim3(256), 0, s, t.diag, t.part, units, t.tiles_m, t.uexp, t.hexp, t.rstats, d,
                     gamma, kap, L_dev, stats_dev);
  BITSMOE_LAUNCH_CHECK("surrogate: finalize launch");
  return ok();
}

extern "C" bitsmoe_status bitsmoe_surrogate_budget(int64_t E, int64_t n_out, int64_t m, int64_t r,
                                                   double b_eq, int64_t* budget_out) {
  if (!budget_out) return fail(BITSMOE_ERR_ARG, "surrogate_budget: null pointer");
  if (E <= 0 || n_out <= 0 || m <= 0 || r <= 0 || r > n_out)
    return fail(BITSMOE_ERR_ARG, "surrogate_budget: sizes must be positive with r <= n_out");
  if (!(b_eq >= 0.0) || !std::isfinite(b_eq)) return fail(BITSMOE_ERR_ARG, "surrogate_budget: b_eq");
  // storage of the projection at b_eq bits per weight minus the fp16 basis,
  // divided by the length of a spectral vector
  const long double total = static_cast<long double>(E) * n_out * m * b_eq;
  const long double basis = 16.0L * n_out * r;
  const long double B = floorl((total - basis) / m);
  if (B < 0.0L) return fail(BITSMOE_ERR_INFEASIBLE, "surrogate_budget: the fp16 basis alone exceeds the budget");
  *budget_out = static_cast<int64_t>(B);
  return ok();
}

extern "C" bitsmoe_status bitsmoe_basis_importance(const float* Vt_dev, int64_t r, int64_t d,
                                                   const float* H_dev, float* beta_dev,
                                                   void* stream) {
  if (!Vt_dev || !H_dev || !beta_dev) return fail(BITSMOE_ERR_ARG, "basis_importance: null pointer");
  if (!aligned16({beta_dev}))
    return fail(BITSMOE_ERR_ARG, "basis_importance: device pointers must be 16-byte aligned");
  bitsmoe_status st = check_rows_args(Vt_dev, H_dev, r, d, "basis_importance");
  if (st != BITSMOE_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  LossTable t;
  st = loss_table_setup(d, r, r, true, stream, "basis_importance", &t);
  if (st != BITSMOE_OK) return st;
  st = loss_table_hoff(H_dev, t, s, "basis_importance: H_off launch");
  if (st != BITSMOE_OK) return st;
  hipLaunchKernelGGL(rowprep_kernel, dim3(static_cast<unsigned>((r + 3) / 4)), dim3(256), 0, s,
                     Vt_dev, r, d, t.hdiag, t.D, t.diag, t.uexp, t.rstats);
  BITSMOE_LAUNCH_CHECK("basis_importance: row launch");
  st = loss_table_gemm(t, stream, "basis_importance", "basis_importance: gemm launch");
  if (st != BITSMOE_OK) return st;
  hipLaunchKernelGGL(quadform_finalize_kernel, dim3(static_cast<unsigned>((r + 255) / 256)),
                     dim3(256), 0, s, t.diag, t.part, r, t.tiles_m, t.uexp, t.hexp, beta_dev);
  BITSMOE_LAUNCH_CHECK("basis_importance: finalize launch");
  return ok();
}

extern "C" bitsmoe_status bitsmoe_score_diag(const float* C_dev, int64_t units, int64_t d,
                                             const float* beta_dev, int64_t r,
                                             const int* bits_host, int nbits, int group,
                                             float* L_dev, void* stream) {
  if (!C_dev || !beta_dev || !bits_host || !L_dev) return fail(BITSMOE_ERR_ARG, "score_diag: null pointer");
  if (!aligned16({C_dev, beta_dev, L_dev}))
    return fail(BITSMOE_ERR_ARG, "score_diag: device pointers must be 16-byte aligned");
  if (units <= 0 || d <= 0 || r <= 0) return fail(BITSMOE_ERR_ARG, "score_diag: non-positive size");
  if (nbits < 1 || nbits > BITSMOE_MAX_NBITS) return fail(BITSMOE_ERR_ARG, "score_diag: nbits outside 1..8");
  QuantBits qb{};
  qb.nb = nbits;
  for (int j = 0; j < nbits; ++j) {
    if (bits_host[j] < 1 || bits_host[j] > BITSMOE_MAX_BITS)
      return fail(BITSMOE_ERR_ARG, "score_diag: width outside 1..8");
    if (j > 0 && bits_host[j] <= bits_host[j - 1])
      return fail(BITSMOE_ERR_ARG, "score_diag: widths must be strictly ascending");
    qb.set(j, bits_host[j]);
  }
  if (!(group == 32 || group == 64 || group == 128 || group == 256))
    return fail(BITSMOE_ERR_SHAPE, "score_diag: group must be 32, 64, 128 or 256");
  if (d % 64 != 0 || d % group != 0)
    return fail(BITSMOE_ERR_SHAPE, "score_diag: d must be a multiple of 64 and of the group");
  if ((units + 3) / 4 > INT32_MAX) return fail(BITSMOE_ERR_SHAPE, "score_diag: too many units");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const unsigned db = static_cast<unsigned>((units + 3) / 4);
  {
    KernelTimer timer("score_diag", stream);
    switch (nbits) {
#define BITSMOE_DNORM(NB)                                                                        \
  case NB:                                                                                       \
    hipLaunchKernelGGL((dgen_kernel<NB, true>), dim3(db), dim3(256), 0, s, C_dev, units, d, group, \
                       qb, nullptr, nullptr, L_dev, nullptr, beta_dev, r);                      \
    break;
      BITSMOE_DNORM(1) BITSMOE_DNORM(2) BITSMOE_DNORM(3) BITSMOE_DNORM(4)
      BITSMOE_DNORM(5) BITSMOE_DNORM(6) BITSMOE_DNORM(7) BITSMOE_DNORM(8)
#undef BITSMOE_DNORM
    }
  }
  BITSMOE_LAUNCH_CHECK("score_diag: launch");
  return ok();
}

extern "C" bitsmoe_status bitsmoe_score_routed(const float* C_dev, int64_t units, int64_t d,
                                               const float* H_dev, int64_t units_per_h,
                                               const int* bits_host, int nbits, int group,
                                               float* L_dev, void* stream) {
  if (!C_dev || !H_dev || !bits_host || !L_dev) return fail(BITSMOE_ERR_ARG, "score_routed: null pointer");
  if (!aligned16({L_dev})) return fail(BITSMOE_ERR_ARG, "score_routed: device pointers must be 16-byte aligned");
  bitsmoe_status st = check_rows_args(C_dev, H_dev, units, d, "score_routed");
  if (st != BITSMOE_OK) return st;
  if (nbits < 1 || nbits > BITSMOE_MAX_NBITS) return fail(BITSMOE_ERR_ARG, "score_routed: nbits outside 1..8");
  QuantBits qb{};
  qb.nb = nbits;
  for (int j = 0; j < nbits; ++j) {
    if (bits_host[j] < 1 || bits_host[j] > BITSMOE_MAX_BITS)
      return fail(BITSMOE_ERR_ARG, "score_routed: width outside 1..8");
    if (j > 0 && bits_host[j] <= bits_host[j - 1])
      return fail(BITSMOE_ERR_ARG, "score_routed: widths must be strictly ascending");
    qb.set(j, bits_host[j]);
  }
  if (!(group == 32 || group == 64 || group == 128 || group == 256))
    return fail(BITSMOE_ERR_SHAPE, "score_routed: group must be 32, 64, 128 or 256");
  if (d % group != 0) return fail(BITSMOE_ERR_SHAPE, "score_routed: d must be a multiple of the group");
  if (units_per_h <= 0 || units % units_per_h != 0)
    return fail(BITSMOE_ERR_SHAPE, "score_routed: units must be a multiple of units_per_h");
  if ((units_per_h * nbits) % SBN != 0)
    return fail(BITSMOE_ERR_SHAPE, "score_routed: units_per_h * nbits must be a multiple of 256");
  const int64_t nh = units / units_per_h;
  if (nh > 65535) return fail(BITSMOE_ERR_SHAPE, "score_routed: too many H matrices");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t R = units * nbits;
  LossTable t;
  st = loss_table_setup(d, R, units, false, stream, "score_routed", &t, nh);
  if (st != BITSMOE_OK) return st;
  st = loss_table_hoff(H_dev, t, s, "score_routed: H_off launch");
  if (st != BITSMOE_OK) return st;
  const unsigned db = static_cast<unsigned>((units + 3) / 4);
  {
    KernelTimer dgen_timer("score_routed_dgen", stream);
    switch (nbits) {
#define BITSMOE_DGEN_R(NB)                                                                       \
  case NB:                                                                                       \
    if (d <= kRowLds)                                                                            \
      hipLaunchKernelGGL((dgen_kernel<NB, false, true>), dim3(db), dim3(256), 0, s, C_dev, units, \
                         d, group, qb, t.hdiag, t.D, t.diag, t.uexp, nullptr, 1, units_per_h);   \
    else                                                                                         \
      hipLaunchKernelGGL((dgen_kernel<NB, false, false>), dim3(db), dim3(256), 0, s, C_dev,      \
                         units, d, group, qb, t.hdiag, t.D, t.diag, t.uexp, nullptr, 1,          \
                         units_per_h);                                                           \
    break;
      BITSMOE_DGEN_R(1) BITSMOE_DGEN_R(2) BITSMOE_DGEN_R(3) BITSMOE_DGEN_R(4)
      BITSMOE_DGEN_R(5) BITSMOE_DGEN_R(6) BITSMOE_DGEN_R(7) BITSMOE_DGEN_R(8)
#undef BITSMOE_DGEN_R
    }
  }
  BITSMOE_LAUNCH_CHECK("score_routed: dgen launch");
  st = loss_table_gemm(t, stream, "score_routed_gemm", "score_routed: gemm launch",
                       units_per_h * nbits);
  if (st != BITSMOE_OK) return st;
  hipLaunchKernelGGL(finalize_kernel, dim3(static_cast<unsigned>((R + 255) / 256)), dim3(256), 0, s,
                     t.diag, t.part, R, t.tiles_m, nbits, t.uexp, t.hexp, L_dev, units_per_h);
  BITSMOE_LAUNCH_CHECK("score_routed: finalize launch");
  return ok();
}
