// Step 3: expert spectral factors C_e = U^T W_e for all experts in one batched
// matrix-core launch.  U is fp32; it is split U = U_hi + U_lo into two bf16
// terms so that the product keeps fp32 accuracy (bf16 W is exact; fp32 W is
// split as well).
#include <algorithm>

#include "bitsmoe.h"
#include "common.hpp"
#include "gemm.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

constexpr int PM = 128;  // basis-vector tile
constexpr int PN = 256;  // input-channel tile
using gemm::BK;

// fp32 -> (hi, lo) bf16, same layout.
__global__ __launch_bounds__(256) void split_f32_kernel(const float* __restrict__ x, int64_t count,
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

// W [E][rows][cols] -> Wt [E][cols][rows] as bf16 (hi, and lo for fp32 input).
template <bool F32>
__global__ __launch_bounds__(256) void batched_transpose_kernel(const void* __restrict__ W,
                                                                int64_t rows, int64_t cols,
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
      hi[in_off + c * rows + r] = h;
      if (F32) lo[in_off + c * rows + r] = f32_to_bf16(v - bf16_to_f32(h));
    }
  }
}

// bf16 W [E][rows][cols] -> Wt [E][cols][rows], 64 x 64 tiles with 16-byte
// loads and stores (rows and cols are multiples of 64).
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ W,
                                                             int64_t rows, int64_t cols,
                                                             uint16_t* __restrict__ Wt) {
  __shared__ __align__(16) uint16_t tile[64][72];  // 144-byte rows: 16-byte aligned, spread over banks
  const int64_t e = blockIdx.z;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * 64;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * 64;
  const int64_t off = e * rows * cols;
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int rr = (t >> 3) + 32 * h, cc = (t & 7) * 8;
    *reinterpret_cast<uint4*>(&tile[rr][cc]) =
        *reinterpret_cast<const uint4*>(W + off + (r0 + rr) * cols + c0 + cc);
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int oc = (t >> 3) + 32 * h;  // output row = input column c0 + oc
    const int orr = (t & 7) * 8;       // first of 8 input rows
    uint16_t v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = tile[orr + i][oc];
    uint4 pk;
    pk.x = v[0] | (static_cast<uint32_t>(v[1]) << 16);
    pk.y = v[2] | (static_cast<uint32_t>(v[3]) << 16);
    pk.z = v[4] | (static_cast<uint32_t>(v[5]) << 16);
    pk.w = v[6] | (static_cast<uint32_t>(v[7]) << 16);
    *reinterpret_cast<uint4*>(Wt + off + (c0 + oc) * rows + r0 + orr) = pk;
  }
}

// C[z][row][col] = acc for row < r, col < d_in.
struct FactorStore {
  float* C;
  int64_t r, d_in;
  template <class F>
  __device__ void operator()(F& f, const gemm::StageLds&) const {
    float* base = C + f.z * r * d_in;
#pragma unroll
    for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
      for (int ni = 0; ni < F::FN; ++ni) {
        const int col = f.col(ni);
        if (col >= d_in) continue;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int row = f.row(mi, q);
          if (row < r) base[static_cast<int64_t>(row) * d_in + col] = f.acc[mi][ni][q];
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
  // scratch A: U hi/lo [2][r][d_out];  scratch B: Wt hi (and lo) [E][d_in][d_out]
  uint16_t* U2 = static_cast<uint16_t*>(scratch(kScratchMisc, 2 * r * d_out * 2, stream, &st));
  if (!U2) return st;
  const int64_t wcount = E * d_out * d_in;
  uint16_t* Wt = static_cast<uint16_t*>(scratch(kScratchB, (f32 ? 2 : 1) * wcount * 2, stream, &st));
  if (!Wt) return st;
  uint16_t* Wt_lo = f32 ? Wt + wcount : nullptr;
  {
    const int64_t count = r * d_out;
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 65536));
    hipLaunchKernelGGL(split_f32_kernel, dim3(blocks), dim3(256), 0, s, Ut_dev, count, U2, U2 + count);
    BITSMOE_LAUNCH_CHECK("project: split launch");
  }
  dim3 tg(static_cast<unsigned>((d_in + 63) / 64), static_cast<unsigned>((d_out + 63) / 64),
          static_cast<unsigned>(E));
  if (f32)
    hipLaunchKernelGGL(batched_transpose_kernel<true>, tg, dim3(256), 0, s, W_dev, d_out, d_in, Wt, Wt_lo);
  else
    hipLaunchKernelGGL(transpose_bf16_kernel, tg, dim3(256), 0, s,
                       static_cast<const uint16_t*>(W_dev), d_out, d_in, Wt);
  BITSMOE_LAUNCH_CHECK("project: transpose launch");

  gemm::Problem p{};
  const uint16_t* Uhi = U2;
  const uint16_t* Ulo = U2 + r * d_out;
  p.a.ld = d_out;
  p.a.rows = r;
  p.a.bstride = 0;
  p.b.ld = d_out;
  p.b.rows = d_in;
  p.b.bstride = d_in * d_out;
  p.segs = 1;
  p.kseg = d_out;
  if (f32) {
    p.passes = 3;  // Uhi*Whi + Uhi*Wlo + Ulo*Whi
    p.a.pass[0] = Uhi; p.b.pass[0] = Wt;
    p.a.pass[1] = Uhi; p.b.pass[1] = Wt_lo;
    p.a.pass[2] = Ulo; p.b.pass[2] = Wt;
  } else {
    p.passes = 2;  // Uhi*W + Ulo*W
    p.a.pass[0] = Uhi; p.b.pass[0] = Wt;
    p.a.pass[1] = Ulo; p.b.pass[1] = Wt;
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
    hipLaunchKernelGGL((gemm::gemm_nt_kernel<PM, PN, 32, 4, FactorStore>), grid,
                       dim3(gemm::kThreads), 0, s, p, epi);
  }
  BITSMOE_LAUNCH_CHECK("project: gemm launch");
  return ok();
}
