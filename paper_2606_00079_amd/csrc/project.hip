// Step 3: expert spectral factors C_e = U^T W_e for all experts in one batched
// matrix-core launch.  U is fp32; it is split U = U_hi + U_lo into two bf16
// terms so that the product keeps fp32 accuracy (bf16 W is exact; fp32 W is
// split as well).  bf16 W is read where it lies: the contraction runs over
// its rows, which the GEMM stages as [32 K][256 N] tiles and reads with the
// transposing LDS read, so no transposed copy is made.
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

// fp32 U^T [r][K] -> (hi, lo) bf16 in the K-tiled layout of PM-row tiles,
// rows padded to r_pad with zeros.
__global__ __launch_bounds__(256) void split_f32_kernel(const float* __restrict__ x, int64_t r,
                                                        int64_t r_pad, int64_t K, int PM,
                                                        uint16_t* __restrict__ hi,
                                                        uint16_t* __restrict__ lo) {
  const int64_t count = r_pad * K;
  const int64_t nkt = K / gemm::kTileK;
  const int64_t TB = static_cast<int64_t>(PM) * gemm::kTileK;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const int64_t t = i / TB, w = i - t * TB;
    const int64_t row = (t / nkt) * PM + w / gemm::kTileK;
    const int64_t k = (t % nkt) * gemm::kTileK + w % gemm::kTileK;
    const float v = row < r ? x[row * K + k] : 0.0f;
    const uint16_t h = f32_to_bf16(v);
    hi[i] = h;
    lo[i] = f32_to_bf16(v - bf16_to_f32(h));
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
// accumulators of a 32 x 32 fragment give each lane one column and 16 rows;
// transposed within each group of four lanes, each lane stores four
// consecutive columns of one row as one 16-byte store (a quarter of the
// store instructions of element-wise stores, whose count bounded the
// epilogue).
struct FactorStore {
  float* C;
  int64_t r, cols;
  template <class F>
  __device__ void operator()(F& f, const gemm::StageLds&) const {
    float* base = C + f.z * r * cols;
    const int k = f.lane & 3;
#pragma unroll
    for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
      for (int ni = 0; ni < F::FN; ++ni) {
        const int c0 = f.col0 + 32 * ni + (f.lane & 28);  // first column of the lane's quad
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float a[4] = {f.acc[mi][ni][4 * j], f.acc[mi][ni][4 * j + 1], f.acc[mi][ni][4 * j + 2],
                        f.acc[mi][ni][4 * j + 3]};
          gemm::quad_transpose(a, k);  // every lane takes part (DPP reads its quad)
          const int row = f.row0 + 32 * mi + 8 * j + 4 * (f.lane >> 5) + k;
          if (row < r && c0 < cols)
            *reinterpret_cast<float4*>(base + static_cast<int64_t>(row) * cols + c0) =
                make_float4(a[0], a[1], a[2], a[3]);
        }
      }
  }
};

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
  // A: U hi/lo, K-tiled [2][r_pad][d_out] (PM-row tiles).  B: bf16 W is read
  // in place as a K-major operand (K = d_out runs over its rows); fp32 W is
  // split into K-tiled transposed hi/lo copies [E][d_in_pad][d_out].
  int PM = 256;
  for (int t : {192, 128})
    if ((r + t - 1) / t * t < (r + PM - 1) / PM * PM) PM = t;
  const int64_t r_pad = (r + PM - 1) / PM * PM;
  const int64_t d_in_pad = (d_in + PN - 1) / PN * PN;
  uint16_t* U2 = static_cast<uint16_t*>(scratch(kScratchMisc, 2 * r_pad * d_out * 2, stream, &st));
  if (!U2) return st;
  {
    const int64_t count = r_pad * d_out;
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 65536));
    hipLaunchKernelGGL(split_f32_kernel, dim3(blocks), dim3(256), 0, s, Ut_dev, r, r_pad, d_out, PM,
                       U2, U2 + count);
    BITSMOE_LAUNCH_CHECK("project: split launch");
  }
  gemm::Problem p{};
  const uint16_t* Uhi = U2;
  const uint16_t* Ulo = U2 + r_pad * d_out;
  static_assert(BK == gemm::kTileK, "the K-tiled operands need the kernel's K step");
  p.a.rows = r_pad;
  p.a.kstep = static_cast<int64_t>(PM) * gemm::kTileK;
  p.a.rtile = static_cast<int64_t>(PM) * d_out;
  p.a.bstride = 0;
  p.segs = 1;
  p.kseg = d_out;
  if (f32) {
    const int64_t wcount = E * d_out * d_in_pad;
    uint16_t* Wt = static_cast<uint16_t*>(scratch(kScratchB, 2 * wcount * 2, stream, &st));
    if (!Wt) return st;
    uint16_t* Wt_lo = Wt + wcount;
    dim3 tg(static_cast<unsigned>((d_in + 63) / 64), static_cast<unsigned>((d_out + 63) / 64),
            static_cast<unsigned>(E));
    hipLaunchKernelGGL(batched_transpose_kernel<true>, tg, dim3(256), 0, s, W_dev, d_out, d_in,
                       d_in_pad, Wt, Wt_lo);
    BITSMOE_LAUNCH_CHECK("project: transpose launch");
    p.b.rows = d_in_pad;
    p.b.kstep = static_cast<int64_t>(PN) * gemm::kTileK;
    p.b.rtile = static_cast<int64_t>(PN) * d_out;
    p.b.bstride = d_in_pad * d_out;
    p.passes = 3;  // Uhi*Whi + Uhi*Wlo + Ulo*Whi
    p.a.pass[0] = Uhi; p.b.pass[0] = Wt;
    p.a.pass[1] = Uhi; p.b.pass[1] = Wt_lo;
    p.a.pass[2] = Ulo; p.b.pass[2] = Wt;
  } else {
    const uint16_t* Wb = static_cast<const uint16_t*>(W_dev);
    p.b.ld = d_in;
    p.b.rows = d_in;  // N extent (columns past it are clamped)
    p.b.kstep = static_cast<int64_t>(gemm::kTileK) * d_in;
    p.b.rtile = PN;
    p.b.bstride = d_out * d_in;
    p.passes = 2;  // Uhi*W + Ulo*W
    p.a.pass[0] = Uhi; p.b.pass[0] = Wb;
    p.a.pass[1] = Ulo; p.b.pass[1] = Wb;
  }
  p.ktiles = static_cast<int64_t>(p.passes) * d_out / BK;
  p.splits = 1;
  p.tiles_m = static_cast<int>((r + PM - 1) / PM);
  p.tiles_n = static_cast<int>((d_in + PN - 1) / PN);
  p.symmetric = 0;
  p.group_n = p.tiles_n;
  FactorStore epi{C_dev, r, d_in};
  dim3 grid(static_cast<unsigned>(p.tiles_m * p.tiles_n), 1, static_cast<unsigned>(E));
  {
    KernelTimer timer("project", stream);
#define BITSMOE_PROJECT(TM, KN)                                                              \
  hipLaunchKernelGGL((gemm::gemm_nt_kernel<TM, PN, 32, 4, FactorStore, false, KN>), grid,   \
                     dim3(gemm::kThreads), 0, s, p, epi)
    if (PM == 256) {
      if (f32) BITSMOE_PROJECT(256, false); else BITSMOE_PROJECT(256, true);
    } else if (PM == 192) {
      if (f32) BITSMOE_PROJECT(192, false); else BITSMOE_PROJECT(192, true);
    } else {
      if (f32) BITSMOE_PROJECT(128, false); else BITSMOE_PROJECT(128, true);
    }
#undef BITSMOE_PROJECT
  }
  BITSMOE_LAUNCH_CHECK("project: gemm launch");
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
    hipLaunchKernelGGL(split_f32_kernel, dim3(blocks), dim3(256), 0, s, Vt_dev, r, r_pad, d_in, PM,
                       V2, V2 + count);
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
  FactorStore epi{C_dev, r, d_out};
  dim3 grid(static_cast<unsigned>(p.tiles_m * p.tiles_n), 1, static_cast<unsigned>(E));
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
