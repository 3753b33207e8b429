// Step 3: expert spectral factors C_e = U^T W_e for all experts in one batched
// matrix-core launch.  bf16 W is read where it lies: the contraction runs
// over its rows, which the GEMM stages as [32 K][256 N] tiles and reads with
// the transposing LDS read, so no transposed copy is made.  It is multiplied
// in one fp16 pass: U (fp32, orthonormal rows) rounded to fp16, each W
// fragment widened from bf16 to fp16 in registers (exact over fp16's range),
// fp32 accumulation: a relative error of about 1.5e-4 in C.  A W entry
// beyond fp16's range makes some factor non-finite, and W entries below
// fp16's normal range (an absolute error of up to 2^-25 each) only matter
// when the factors are small too; the epilogue flags either case and a
// second launch, which otherwise returns at once, recomputes C with the
// exact two-pass form U = U_hi + U_lo in bf16.  fp32 W (split into hi and
// lo as well) takes three bf16 passes.
#include <algorithm>

#include "bitsmoe.h"
#include "common.hpp"
#include "gemm.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

// Basis-vector tile: 256, 192 or 128 rows, the largest that pads r least
// (taller tiles read fewer LDS fragments per matrix-core op).
constexpr int PN = 256;  // input-channel tile
using gemm::BK;

// fp32 U^T [r][K] in the K-tiled layout of PM-row tiles (rows padded to
// r_pad with zeros), as bf16 hi + lo planes (x ~ hi + lo to 2^-16):
//   FOR_F16 = false: hi, then lo (lo = hi + r_pad K), two K-tiled matrices;
//   FOR_F16 = true:  the fp16 rounding of x (one K-tiled matrix, first), then
//                    one K-tiled matrix of 2K columns whose K tile 2q is the
//                    hi part and 2q + 1 the lo part of K tile q (the exact
//                    two-pass form with the terms of a K tile back to back),
//                    and thread 0 clears *flag.
template <bool FOR_F16>
__global__ __launch_bounds__(256) void split_f32_kernel(const float* __restrict__ x, int64_t r,
                                                        int64_t r_pad, int64_t K, int PM,
                                                        uint16_t* __restrict__ out,
                                                        int* __restrict__ flag) {
  const int64_t count = r_pad * K;
  const int64_t nkt = K / gemm::kTileK;
  const int64_t TB = static_cast<int64_t>(PM) * gemm::kTileK;
  if (FOR_F16 && blockIdx.x == 0 && threadIdx.x == 0) *flag = 0;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const int64_t t = i / TB, w = i - t * TB;
    const int64_t rt = t / nkt, kt = t % nkt;
    const int64_t row = rt * PM + w / gemm::kTileK;
    const int64_t k = kt * gemm::kTileK + w % gemm::kTileK;
    const float v = row < r ? x[row * K + k] : 0.0f;
    const uint16_t h = f32_to_bf16(v);
    const uint16_t l = f32_to_bf16(v - bf16_to_f32(h));
    if (FOR_F16) {
      out[i] = f32_to_f16_bits(v);
      uint16_t* il = out + count;
      const int64_t o = (rt * 2 * nkt + 2 * kt) * TB + w;
      il[o] = h;
      il[o + TB] = l;
    } else {
      out[i] = h;
      out[i + count] = l;
    }
  }
}

// W [E][rows][cols] -> Wt [E][cols_pad][rows] as bf16 (hi, and lo for fp32
// input), K-tiled with PN-row tiles (rows of Wt = columns of W; K = rows).
template <bool F32>
__global__ __launch_bounds__(256) void batched_transpose_kernel(const void* __restrict__ W,
                                                                int64_t rows, int64_t cols,
                                                                int64_t cols_pad,
                                                                uint16_t* __restrict__ hi,
                                                                uint16_t* __restrict__ lo) {
  __shared__ float tile[64][65];
  const int64_t e = blockIdx.z;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * 64;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t in_off = e * rows * cols;
  for (int i = ty; i < 64; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    float v = 0.0f;
    if (r < rows && c < cols) {
      if (F32)
        v = static_cast<const float*>(W)[in_off + r * cols + c];
      else
        v = bf16_to_f32(static_cast<const uint16_t*>(W)[in_off + r * cols + c]);
    }
    tile[i][tx] = v;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) {
      const float v = tile[tx][i];
      const uint16_t h = f32_to_bf16(v);
      const int64_t o = e * cols_pad * rows + gemm::tiled_offset(c, r, rows, PN);
      hi[o] = h;
      if (F32) lo[o] = f32_to_bf16(v - bf16_to_f32(h));
    }
  }
}

// fp32 x -> (hi, lo) bf16, element by element (row-major operands).
__global__ __launch_bounds__(256) void split_rows_kernel(const float* __restrict__ x, int64_t count,
                                                         uint16_t* __restrict__ hi,
                                                         uint16_t* __restrict__ lo) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const float v = x[i];
    const uint16_t h = f32_to_bf16(v);
    hi[i] = h;
    lo[i] = f32_to_bf16(v - bf16_to_f32(h));
  }
}

// C[z][row][col] = acc for row < r, col < cols (cols a multiple of 4).  The
// accumulators of a 32 x 32 fragment give each lane one column and 16 rows.
// A wave whose block lies wholly inside C stores them element by element
// through a buffer resource (store_full); one partly outside transposes them
// within each group of four lanes, so that each lane stores four consecutive
// columns of one row as one bounds-tested 16-byte store.
// With `inexact` set (the one-pass fp16 form), a wave writes 1 there when a
// factor it stores is not finite (a W entry beyond fp16's range comes out
// infinite) or when every factor it stores is below kSmallFactor in
// magnitude (W entries below fp16's normal range carry an absolute error of
// up to 2^-25 each, which only matters against factors that small); the
// flag asks for the exact two-pass form.
constexpr float kSmallFactor = 0.015625f;  // 2^-6
struct FactorStore {
  static constexpr bool kUsesLds = false;  // reads or writes the stage buffers
  float* C;
  int64_t r, cols;
  int* inexact;
  template <class F>
  __device__ void operator()(F& f, const gemm::StageLds&) const {
    // the lane index made opaque: no address arithmetic of the stores is
    // hoisted into the K loop (where it would hold registers throughout)
    const int lane = opaque(f.lane);
    float* base = C + f.z * r * cols;
    // (rows of at most 2^20 columns: the block's byte offsets fit 31 bits)
    if (f.row0 + F::WM <= r && f.col0 + F::WN <= cols &&
        cols <= (int64_t{1} << 20)) {
      store_full(f, lane, base);
      return;
    }
    const int k = lane & 3;
    bool bad = false, stored = false, big = false;
#pragma unroll
    for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
      for (int ni = 0; ni < F::FN; ++ni) {
        const int c0 = f.col0 + 32 * ni + (lane & 28);  // first column of the lane's quad
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float a[4] = {f.acc[mi][ni][4 * j], f.acc[mi][ni][4 * j + 1], f.acc[mi][ni][4 * j + 2],
                        f.acc[mi][ni][4 * j + 3]};
          gemm::quad_transpose(a, k);  // every lane takes part (DPP reads its quad)
          const int row = f.row0 + 32 * mi + 8 * j + 4 * (lane >> 5) + k;
          if (row < r && c0 < cols) {
            *reinterpret_cast<float4*>(base + static_cast<int64_t>(row) * cols + c0) =
                make_float4(a[0], a[1], a[2], a[3]);
            if (inexact) {
              const float m = fmaxf(fmaxf(fabsf(a[0]), fabsf(a[1])), fmaxf(fabsf(a[2]), fabsf(a[3])));
              // m <= max finite is false for inf and nan (fmaxf drops a nan
              // only next to a number, so test every entry as well)
              bad |= !(m <= 3.4e38f) || a[0] != a[0] || a[1] != a[1] || a[2] != a[2] || a[3] != a[3];
              big |= m >= kSmallFactor;
              stored = true;
            }
          }
        }
      }
    if (inexact && (__any(bad) || (__any(stored) && !__any(big))) && lane == 0) *inexact = 1;
  }

  // The wave's whole WM x WN block lies inside C (wave-uniform test): every
  // accumulator goes out as one 4-byte store, those of one register of the
  // 64 lanes covering 32 columns of two rows (two whole 128-byte lines).
  // Through a buffer resource at the block's origin the lane's offset stays
  // fixed and the row is the scalar offset: no address arithmetic, bounds
  // test or lane exchange per store.  The inexact test runs on the largest
  // magnitude, taken with NaN-propagating maxima.
  template <class F>
  __device__ void store_full(F& f, int lane, float* base) const {
    float* wbase = base + static_cast<int64_t>(f.row0) * cols + f.col0;
    const int64_t left = (r - f.row0) * cols - f.col0;  // elements from wbase to the end of C_z
    const int nrec = static_cast<int>(left < (int64_t{1} << 29) ? left * 4 : (int64_t{1} << 31) - 4);
    // raw buffer (stride 0: num_records counts bytes, accesses past it are
    // dropped); word 3 0x00020000 = 32-bit data format, the value for plain
    // dword buffer loads and stores on this architecture
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(wbase, static_cast<short>(0), nrec, 0x00020000);
    const int vo = ((4 * (lane >> 5)) * static_cast<int>(cols) + (lane & 31)) * 4;
    const int rowb = static_cast<int>(cols) * 4;  // bytes per row
    float m = 0.0f;
#pragma unroll
    for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
      for (int ni = 0; ni < F::FN; ++ni)
#pragma unroll
        for (int q = 0; q < 16; q += 2) {
          const float v0 = f.acc[mi][ni][q], v1 = f.acc[mi][ni][q + 1];
          const int row = 32 * mi + 8 * (q >> 2) + (q & 3);
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v0), rs, vo + 128 * ni, row * rowb, 0);
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v1), rs, vo + 128 * ni, (row + 1) * rowb, 0);
          if (inexact)
            m = __builtin_elementwise_maximum(
                m, __builtin_elementwise_maximum(__builtin_fabsf(v0), __builtin_fabsf(v1)));
        }
    if (inexact) {
      const bool bad = !(m <= 3.4e38f);  // NaN or infinity
      const bool big = m >= kSmallFactor;
      if ((__any(bad) || !__any(big)) && lane == 0) *inexact = 1;
    }
  }
};

// Launch grid of a factor GEMM over E experts of p.flat tiles each: for a
// one-pass, one-segment problem with more tiles than compute units (and
// `persistent`), one persistent workgroup per compute unit
// (a multiple of the XCD count) walks its XCD's tiles in turn, issuing each
// next tile's first loads ahead of the current tile's stores; otherwise one
// workgroup per tile.
dim3 factor_grid(gemm::Problem& p, int64_t E, bool persistent) {
  const int64_t n = static_cast<int64_t>(p.flat) * E;
  const int64_t g = device_cus() / gemm::kXcds * gemm::kXcds;
  if (persistent && p.passes == 1 && p.segs == 1 && g >= gemm::kXcds && n > g) {
    p.persist = n;
    return dim3(static_cast<unsigned>(g), 1, 1);
  }
  p.persist = 0;
  return dim3(static_cast<unsigned>(n), 1, 1);
}

}  // namespace
}  // namespace bitsmoe

using namespace bitsmoe;

extern "C" bitsmoe_status bitsmoe_project(const float* Ut_dev, const void* W_dev, bitsmoe_dtype wt,
                                          int64_t E, int64_t d_out, int64_t d_in, int64_t r,
                                          float* C_dev, void* stream) {
  if (!Ut_dev || !W_dev || !C_dev) return fail(BITSMOE_ERR_ARG, "project: null pointer");
  if (!aligned16({Ut_dev, W_dev, C_dev}))
    return fail(BITSMOE_ERR_ARG, "project: device pointers must be 16-byte aligned");
  if (E <= 0 || d_out <= 0 || d_in <= 0 || r <= 0) return fail(BITSMOE_ERR_ARG, "project: non-positive size");
  if (wt != BITSMOE_F32 && wt != BITSMOE_BF16) return fail(BITSMOE_ERR_DTYPE, "project: dtype");
  if (d_out % 64 != 0 || d_in % 64 != 0)
    return fail(BITSMOE_ERR_SHAPE, "project: d_out and d_in must be multiples of 64");
  if (r > d_out) return fail(BITSMOE_ERR_SHAPE, "project: r > d_out");
  if (E > 65535) return fail(BITSMOE_ERR_SHAPE, "project: too many experts");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool f32 = wt == BITSMOE_F32;
  bitsmoe_status st;
  // Tile: PM rows of U^T (the size that pads r least) x PN columns of W.
  int PM = 256;
  for (int t : {192, 128})
    if ((r + t - 1) / t * t < (r + PM - 1) / PM * PM) PM = t;
  const int64_t r_pad = (r + PM - 1) / PM * PM;
  const int64_t d_in_pad = (d_in + PN - 1) / PN * PN;
  const int64_t ucount = r_pad * d_out;
  // small tables: a flag (256 bytes), then U as fp16 (bf16 W) and as bf16
  // hi/lo planes
  char* misc = static_cast<char*>(scratch(kScratchMisc, 256 + 3 * ucount * 2, stream, &st));
  if (!misc) return st;
  int* flag = reinterpret_cast<int*>(misc);
  uint16_t* U16 = reinterpret_cast<uint16_t*>(misc + 256);
  {
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((ucount + 255) / 256, 65536));
    if (f32)
      hipLaunchKernelGGL(split_f32_kernel<false>, dim3(blocks), dim3(256), 0, s, Ut_dev, r, r_pad,
                         d_out, PM, U16, flag);
    else
      hipLaunchKernelGGL(split_f32_kernel<true>, dim3(blocks), dim3(256), 0, s, Ut_dev, r, r_pad,
                         d_out, PM, U16, flag);
    BITSMOE_LAUNCH_CHECK("project: split launch");
  }
  static_assert(BK == gemm::kTileK, "the K-tiled operands need the kernel's K step");
  gemm::Problem p{};
  p.a.rows = r_pad;
  p.a.kstep = static_cast<int64_t>(PM) * gemm::kTileK;
  p.a.rtile = static_cast<int64_t>(PM) * d_out;
  p.segs = 1;
  p.kseg = d_out;
  p.splits = 1;
  p.tiles_m = static_cast<int>((r + PM - 1) / PM);
  p.tiles_n = static_cast<int>((d_in + PN - 1) / PN);
  p.group_n = p.tiles_n;
  // XCD-aware grid: an expert's tiles run together on one XCD, so its W is
  // fetched into that XCD's L2 once for all of them
  p.flat = p.tiles_m * p.tiles_n;
  KernelTimer timer("project", stream);
  if (f32) {
    // fp32 W: transposed K-tiled hi/lo copies, three bf16 passes
    const int64_t wcount = E * d_out * d_in_pad;
    uint16_t* Wt = static_cast<uint16_t*>(scratch(kScratchB, 2 * wcount * 2, stream, &st));
    if (!Wt) return st;
    uint16_t* Wt_lo = Wt + wcount;
    dim3 tg(static_cast<unsigned>((d_in + 63) / 64), static_cast<unsigned>((d_out + 63) / 64),
            static_cast<unsigned>(E));
    hipLaunchKernelGGL(batched_transpose_kernel<true>, tg, dim3(256), 0, s, W_dev, d_out, d_in,
                       d_in_pad, Wt, Wt_lo);
    BITSMOE_LAUNCH_CHECK("project: transpose launch");
    const uint16_t* Uhi = U16;
    const uint16_t* Ulo = U16 + ucount;
    p.b.rows = d_in_pad;
    p.b.kstep = static_cast<int64_t>(PN) * gemm::kTileK;
    p.b.rtile = static_cast<int64_t>(PN) * d_out;
    p.b.bstride = d_in_pad * d_out;
    p.passes = 3;  // Uhi*Whi + Uhi*Wlo + Ulo*Whi
    p.a.pass[0] = Uhi; p.b.pass[0] = Wt;
    p.a.pass[1] = Uhi; p.b.pass[1] = Wt_lo;
    p.a.pass[2] = Ulo; p.b.pass[2] = Wt;
    p.ktiles = 3 * d_out / BK;
    const dim3 grid = factor_grid(p, E, false);
    FactorStore epi{C_dev, r, d_in, nullptr};
#define BITSMOE_PROJECT3(TM)                                                                   \
  hipLaunchKernelGGL((gemm::gemm_nt_kernel<TM, PN, 32, 4, FactorStore>), grid,                \
                     dim3(gemm::kThreads), 0, s, p, epi)
    if (PM == 256) BITSMOE_PROJECT3(256); else if (PM == 192) BITSMOE_PROJECT3(192); else BITSMOE_PROJECT3(128);
#undef BITSMOE_PROJECT3
    BITSMOE_LAUNCH_CHECK("project: gemm launch");
    return ok();
  }
  // bf16 W is read where it lies as a K-major operand (K = d_out runs over
  // its rows).  One pass: U rounded to fp16 (relative error <= 2^-12), each
  // W fragment widened to fp16 in registers (exact for |W| in 2^-14 ..
  // 65504), fp32 accumulation.
  const uint16_t* Wb = static_cast<const uint16_t*>(W_dev);
  p.b.ld = d_in;
  p.b.rows = d_in;  // N extent (columns past it are clamped)
  p.b.kstep = static_cast<int64_t>(gemm::kTileK) * d_in;
  p.b.rtile = PN;
  p.b.bstride = d_out * d_in;
  p.passes = 1;
  p.a.pass[0] = U16; p.b.pass[0] = Wb;
  p.ktiles = d_out / BK;
  {
    // persistent for the 192- and 128-row tiles (the 256-row persistent
    // kernel does not fit the register file without spilling)
    const dim3 grid = factor_grid(p, E, PM != 256);
    FactorStore epi{C_dev, r, d_in, flag};
    // one pass, one segment: the minimal K walk (ONEK)
    // the four waves side by side along N (each all TM rows of U^T and 64
    // columns of W): every W fragment is read and widened by one wave, not
    // two as with 2 x 2 waves, for a quarter more fragment reads of U^T
#define BITSMOE_PROJECT16(TM, PERSIST)                                                            \
  hipLaunchKernelGGL((gemm::gemm_nt_kernel<TM, PN, 32, 4, FactorStore, true, true, false, true,      \
                                           PERSIST, true, 4>), grid, dim3(gemm::kThreads), 0, s, p, epi)
    if (PM == 256)
      BITSMOE_PROJECT16(256, false);
    else if (PM == 192 && p.persist)
      BITSMOE_PROJECT16(192, true);
    else if (PM == 192)
      BITSMOE_PROJECT16(192, false);
    else if (p.persist)
      BITSMOE_PROJECT16(128, true);
    else
      BITSMOE_PROJECT16(128, false);
#undef BITSMOE_PROJECT16
    BITSMOE_LAUNCH_CHECK("project: gemm launch");
  }
  // Only if the one-pass form flagged a tile (a non-finite factor: a W entry
  // beyond fp16's range, or a non-finite input; or a tile of factors all
  // below 2^-6): the exact two-pass bf16 form, U = hi + lo, the
  // two terms of a K tile back to back (d_out / 32 segments of two K tiles;
  // A advances a tile at a time through the interleaved planes, B stays on
  // the segment's K tile, so W's second read of a tile hits L2).  Otherwise
  // its workgroups return at once.
  p.a.pass[0] = U16 + ucount;
  p.a.rtile = static_cast<int64_t>(PM) * 2 * d_out;
  p.a.estride = 2 * p.a.kstep;
  p.b.estride = p.b.kstep;
  p.b.repeat_k = 1;
  p.segs = static_cast<int>(d_out / gemm::kTileK);
  p.kseg = 2 * gemm::kTileK;
  p.ktiles = 2 * d_out / BK;
  p.run_if = flag;
  {
    const dim3 grid = factor_grid(p, E, false);
    FactorStore epi{C_dev, r, d_in, nullptr};
#define BITSMOE_PROJECT2(TM)                                                                    \
  hipLaunchKernelGGL((gemm::gemm_nt_kernel<TM, PN, 32, 4, FactorStore, false, true>), grid,      \
                     dim3(gemm::kThreads), 0, s, p, epi)
    if (PM == 256) BITSMOE_PROJECT2(256); else if (PM == 192) BITSMOE_PROJECT2(192); else BITSMOE_PROJECT2(128);
#undef BITSMOE_PROJECT2
    BITSMOE_LAUNCH_CHECK("project: exact gemm launch");
  }
  return ok();
}

// Input-space factors of the gate/up projections: C_e = Phi_r^T W_e^T, i.e.
// acc[k][j] = sum_i Vt[k][i] W_e[j][i]; both operands are contiguous along
// K = d_in, so W is read row-major where it lies (fp32 W split into hi/lo).
extern "C" bitsmoe_status bitsmoe_project_in(const float* Vt_dev, const void* W_dev,
                                             bitsmoe_dtype wt, int64_t E, int64_t d_out,
                                             int64_t d_in, int64_t r, float* C_dev, void* stream) {
  if (!Vt_dev || !W_dev || !C_dev) return fail(BITSMOE_ERR_ARG, "project_in: null pointer");
  if (!aligned16({Vt_dev, W_dev, C_dev}))
    return fail(BITSMOE_ERR_ARG, "project_in: device pointers must be 16-byte aligned");
  if (E <= 0 || d_out <= 0 || d_in <= 0 || r <= 0)
    return fail(BITSMOE_ERR_ARG, "project_in: non-positive size");
  if (wt != BITSMOE_F32 && wt != BITSMOE_BF16) return fail(BITSMOE_ERR_DTYPE, "project_in: dtype");
  if (d_out % 64 != 0 || d_in % 64 != 0)
    return fail(BITSMOE_ERR_SHAPE, "project_in: d_out and d_in must be multiples of 64");
  if (r > d_in) return fail(BITSMOE_ERR_SHAPE, "project_in: r > d_in");
  if (E > 65535) return fail(BITSMOE_ERR_SHAPE, "project_in: too many experts");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool f32 = wt == BITSMOE_F32;
  bitsmoe_status st;
  int PM = 256;
  for (int t : {192, 128})
    if ((r + t - 1) / t * t < (r + PM - 1) / PM * PM) PM = t;
  const int64_t r_pad = (r + PM - 1) / PM * PM;
  uint16_t* V2 = static_cast<uint16_t*>(scratch(kScratchMisc, 2 * r_pad * d_in * 2, stream, &st));
  if (!V2) return st;
  {
    const int64_t count = r_pad * d_in;
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 65536));
    hipLaunchKernelGGL(split_f32_kernel<false>, dim3(blocks), dim3(256), 0, s, Vt_dev, r, r_pad,
                       d_in, PM, V2, nullptr);
    BITSMOE_LAUNCH_CHECK("project_in: split launch");
  }
  gemm::Problem p{};
  const uint16_t* Vhi = V2;
  const uint16_t* Vlo = V2 + r_pad * d_in;
  p.a.rows = r_pad;
  p.a.kstep = static_cast<int64_t>(PM) * gemm::kTileK;
  p.a.rtile = static_cast<int64_t>(PM) * d_in;
  p.a.bstride = 0;
  p.b.ld = d_in;
  p.b.rows = d_out;  // rows past it are clamped
  p.b.kstep = 0;     // row-major
  p.b.bstride = d_out * d_in;
  p.segs = 1;
  p.kseg = d_in;
  const uint16_t* Wb = static_cast<const uint16_t*>(W_dev);
  if (f32) {
    const int64_t wcount = E * d_out * d_in;
    uint16_t* W2 = static_cast<uint16_t*>(scratch(kScratchB, 2 * wcount * 2, stream, &st));
    if (!W2) return st;
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((wcount + 255) / 256, 65536));
    hipLaunchKernelGGL(split_rows_kernel, dim3(blocks), dim3(256), 0, s,
                       static_cast<const float*>(W_dev), wcount, W2, W2 + wcount);
    BITSMOE_LAUNCH_CHECK("project_in: W split launch");
    p.passes = 3;  // Vhi*Whi + Vhi*Wlo + Vlo*Whi
    p.a.pass[0] = Vhi; p.b.pass[0] = W2;
    p.a.pass[1] = Vhi; p.b.pass[1] = W2 + wcount;
    p.a.pass[2] = Vlo; p.b.pass[2] = W2;
  } else {
    p.passes = 2;  // Vhi*W + Vlo*W
    p.a.pass[0] = Vhi; p.b.pass[0] = Wb;
    p.a.pass[1] = Vlo; p.b.pass[1] = Wb;
  }
  p.ktiles = static_cast<int64_t>(p.passes) * d_in / BK;
  p.splits = 1;
  p.tiles_m = static_cast<int>((r + PM - 1) / PM);
  p.tiles_n = static_cast<int>((d_out + PN - 1) / PN);
  p.symmetric = 0;
  p.group_n = p.tiles_n;
  p.flat = p.tiles_m * p.tiles_n;  // XCD-aware grid, as in bitsmoe_project
  FactorStore epi{C_dev, r, d_out, nullptr};
  const dim3 grid = factor_grid(p, E, false);
  {
    KernelTimer timer("project_in", stream);
#define BITSMOE_PROJECT_IN(TM)                                                                \
  hipLaunchKernelGGL((gemm::gemm_nt_kernel<TM, PN, 32, 4, FactorStore>), grid,                \
                     dim3(gemm::kThreads), 0, s, p, epi)
    if (PM == 256)
      BITSMOE_PROJECT_IN(256);
    else if (PM == 192)
      BITSMOE_PROJECT_IN(192);
    else
      BITSMOE_PROJECT_IN(128);
#undef BITSMOE_PROJECT_IN
  }
  BITSMOE_LAUNCH_CHECK("project_in: gemm launch");
  return ok();
}
