// Step 1: the calibration Gram H = X^T X / n and the cross-expert Gram
// M = sum_e W_e W_e^T, both as symmetric split-K matrix-core GEMMs whose fp32
// partial tiles are added in fp64 in a fixed order (deterministic).
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <string>

#include "bitsmoe.h"
#include "common.hpp"
#include "gemm.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

constexpr int GT = 256;  // tile edge of the symmetric GEMMs
using gemm::BK;

// X [n][d] -> Xt [d_pad][npad] (bf16) in the K-tiled layout of GT-row tiles
// (K = tokens), tokens beyond n zero.  For fp32 input the value is split
// x = hi + lo with hi = bf16(x), lo = bf16(x - hi).
template <bool F32>
__global__ __launch_bounds__(256) void transpose_split_kernel(const void* __restrict__ X, int64_t n,
                                                              int64_t d, int64_t npad,
                                                              uint16_t* __restrict__ hi,
                                                              uint16_t* __restrict__ lo) {
  __shared__ float tile[64][65];
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * 64;  // token block
  const int64_t c0 = static_cast<int64_t>(blockIdx.y) * 64;  // channel block
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;     // 64 x 4
  for (int i = ty; i < 64; i += 4) {
    const int64_t t = t0 + i, c = c0 + tx;
    float v = 0.0f;
    if (t < n && c < d) {
      if (F32)
        v = static_cast<const float*>(X)[t * d + c];
      else
        v = bf16_to_f32(static_cast<const uint16_t*>(X)[t * d + c]);
    }
    tile[i][tx] = v;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, t = t0 + tx;
    if (c < d && t < npad) {
      const float v = tile[tx][i];
      const uint16_t h = f32_to_bf16(v);
      const int64_t o = gemm::tiled_offset(c, t, npad, GT);
      hi[o] = h;
      if (F32) lo[o] = f32_to_bf16(v - bf16_to_f32(h));
    }
  }
}

// fp32 W -> (hi, lo) bf16 with the same layout.
__global__ __launch_bounds__(256) void split_kernel(const float* __restrict__ W, int64_t count,
                                                    uint16_t* __restrict__ hi,
                                                    uint16_t* __restrict__ lo) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const float v = W[i];
    const uint16_t h = f32_to_bf16(v);
    hi[i] = h;
    lo[i] = f32_to_bf16(v - bf16_to_f32(h));
  }
}

// Routed rows of expert e = blockIdx.z, in the K-tiled layout of the
// symmetric GEMM (rows = channels, K = the expert's tokens, zero-padded to
// npad): the A side holds x_{rows[i]} (fp32 input split into bf16 hi + lo),
// the B side w_i x_{rows[i]} split into hi + lo.  Routing entries are
// checked on the host (rows in [0, n)).
template <bool F32>
__global__ __launch_bounds__(256) void routed_gather_kernel(
    const void* __restrict__ X, int64_t d, const int64_t* __restrict__ off,
    const int32_t* __restrict__ rows, const float* __restrict__ w, int64_t npad, int64_t d_pad,
    uint16_t* __restrict__ a_hi, uint16_t* __restrict__ a_lo, uint16_t* __restrict__ b_hi,
    uint16_t* __restrict__ b_lo) {
  __shared__ float tile[64][65];
  __shared__ float wt[64];
  const int64_t e = blockIdx.z;
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * 64;  // token block of the expert
  const int64_t c0 = static_cast<int64_t>(blockIdx.y) * 64;  // channel block
  const int64_t o0 = off[e], ne = off[e + 1] - o0;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  if (ty == 0) wt[tx] = (i0 + tx < ne) ? w[o0 + i0 + tx] : 0.0f;
  for (int i = ty; i < 64; i += 4) {
    const int64_t t = i0 + i, c = c0 + tx;
    float v = 0.0f;
    if (t < ne && c < d) {
      const int64_t row = rows[o0 + t];
      if (F32)
        v = static_cast<const float*>(X)[row * d + c];
      else
        v = bf16_to_f32(static_cast<const uint16_t*>(X)[row * d + c]);
    }
    tile[i][tx] = v;
  }
  __syncthreads();
  const int64_t base = e * d_pad * npad;
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, t = i0 + tx;
    if (c < d) {
      const float v = tile[tx][i];
      const int64_t o = base + gemm::tiled_offset(c, t, npad, GT);
      const uint16_t h = f32_to_bf16(v);
      a_hi[o] = h;
      if (F32) a_lo[o] = f32_to_bf16(v - bf16_to_f32(h));
      const float wv = wt[tx] * v;
      const uint16_t hb = f32_to_bf16(wv);
      b_hi[o] = hb;
      b_lo[o] = f32_to_bf16(wv - bf16_to_f32(hb));
    }
  }
}

// Stores each wave's fp32 accumulators into partials[batch][split][tile][GT][GT].
struct PartialStore {
  static constexpr bool kUsesLds = false;  // reads or writes the stage buffers
  float* part;
  int64_t ntiles;     // tiles in the upper triangle
  int ntiles_side;    // tiles per side
  int64_t zstride;    // elements per batch (splits * ntiles * GT * GT)
  template <class F>
  __device__ void operator()(F& f, const gemm::StageLds&) const {
    const int64_t t = (static_cast<int64_t>(f.tm) * (2 * ntiles_side - f.tm + 1)) / 2 + (f.tn - f.tm);
    float* base = part + f.z * zstride + (static_cast<int64_t>(f.ks) * ntiles + t) * GT * GT;
    // four consecutive columns of one row per lane and 16-byte store (the
    // fragment's columns transposed within each group of four lanes)
    const int k = f.lane & 3;
#pragma unroll
    for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
      for (int ni = 0; ni < F::FN; ++ni) {
        const int lc0 = f.col0 - f.tn * GT + 32 * ni + (f.lane & 28);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float a[4] = {f.acc[mi][ni][4 * j], f.acc[mi][ni][4 * j + 1], f.acc[mi][ni][4 * j + 2],
                        f.acc[mi][ni][4 * j + 3]};
          gemm::quad_transpose(a, k);
          const int lr = f.row0 - f.tm * GT + 32 * mi + 8 * j + 4 * (f.lane >> 5) + k;
          *reinterpret_cast<float4*>(base + lr * GT + lc0) = make_float4(a[0], a[1], a[2], a[3]);
        }
      }
  }
};

// out = scale * sum over splits of the partial tiles (fp64, splits in
// order), mirrored into the lower triangle.  One workgroup per 16 x 64 block
// of an upper-triangle tile; a thread owns four adjacent columns of one row
// and keeps eight splits' loads in flight before adding them in order.
// Blocks of off-diagonal tiles are also written transposed through LDS.
constexpr int RB_ROWS = 16;
constexpr int RB_COLS = 64;
constexpr int RB_UNROLL = 8;

__device__ __forceinline__ void store4(double* p, const double (&v)[4]) {
  reinterpret_cast<double2*>(p)[0] = make_double2(v[0], v[1]);
  reinterpret_cast<double2*>(p)[1] = make_double2(v[2], v[3]);
}
__device__ __forceinline__ void store4(float* p, const double (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(static_cast<float>(v[0]), static_cast<float>(v[1]),
                                              static_cast<float>(v[2]), static_cast<float>(v[3]));
}

template <typename OutT>
__global__ __launch_bounds__(256) void sym_reduce_kernel(const float* __restrict__ part, int splits,
                                                         int64_t ntiles, int T, int64_t d,
                                                         double scale, OutT* __restrict__ out) {
  __shared__ double tile[RB_ROWS][RB_COLS + 1];
  // batch blockIdx.y: its own partials and output matrix
  part += static_cast<int64_t>(blockIdx.y) * splits * ntiles * GT * GT;
  out += static_cast<int64_t>(blockIdx.y) * d * d;
  constexpr int SR = GT / RB_ROWS, SC = GT / RB_COLS;  // blocks per tile edge
  const int64_t t = blockIdx.x / (SR * SC);            // upper-triangle tile
  const int sb = static_cast<int>(blockIdx.x % (SR * SC));
  int tm = 0, rem = static_cast<int>(t);
  while (rem >= T - tm) {
    rem -= T - tm;
    ++tm;
  }
  const int tn = tm + rem;
  const int bi = sb / SC, bj = sb % SC;
  const int64_t gi0 = static_cast<int64_t>(tm) * GT + RB_ROWS * bi;  // first output row
  const int64_t gj0 = static_cast<int64_t>(tn) * GT + RB_COLS * bj;  // first output column
  // d is a multiple of 64, so a block is either wholly inside or wholly outside
  if (gi0 >= d || gj0 >= d) return;
  const int r = threadIdx.x >> 4, cq = threadIdx.x & 15;
  const float* src = part + t * GT * GT + static_cast<int64_t>(RB_ROWS * bi + r) * GT + RB_COLS * bj + 4 * cq;
  const int64_t kstride = ntiles * GT * GT;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  int k = 0;
  for (; k + RB_UNROLL <= splits; k += RB_UNROLL) {
    float4 v[RB_UNROLL];
#pragma unroll
    for (int u = 0; u < RB_UNROLL; ++u) v[u] = *reinterpret_cast<const float4*>(src + (k + u) * kstride);
#pragma unroll
    for (int u = 0; u < RB_UNROLL; ++u) {
      acc[0] += static_cast<double>(v[u].x);
      acc[1] += static_cast<double>(v[u].y);
      acc[2] += static_cast<double>(v[u].z);
      acc[3] += static_cast<double>(v[u].w);
    }
  }
  for (; k < splits; ++k) {
    const float4 v = *reinterpret_cast<const float4*>(src + k * kstride);
    acc[0] += static_cast<double>(v.x);
    acc[1] += static_cast<double>(v.y);
    acc[2] += static_cast<double>(v.z);
    acc[3] += static_cast<double>(v.w);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] *= scale;
  if (tm == tn) {
    // a diagonal tile holds both triangles; its upper one is written and
    // mirrored, so the output is exactly symmetric even when the two GEMM
    // operands differ in rounding (the routed Gram's weighted side)
    const int64_t row = gi0 + r;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t col = gj0 + 4 * cq + j;
      if (col >= row) out[row * d + col] = static_cast<OutT>(acc[j]);
      if (col > row) out[col * d + row] = static_cast<OutT>(acc[j]);
    }
    return;
  }
  store4(out + (gi0 + r) * d + gj0 + 4 * cq, acc);
#pragma unroll
  for (int j = 0; j < 4; ++j) tile[r][4 * cq + j] = acc[j];
  __syncthreads();
  // transposed: output row gj0 + c, columns gi0 + 4q .. 4q + 3
  const int c = threadIdx.x >> 2, q = threadIdx.x & 3;
  const double tv[4] = {tile[4 * q][c], tile[4 * q + 1][c], tile[4 * q + 2][c], tile[4 * q + 3][c]};
  store4(out + (gj0 + c) * d + gi0 + 4 * q, tv);
}

// Launches the symmetric split-K GEMM of p (tiles/splits already set) and
// reduces it into out.
// `batches` independent problems (blockIdx.z, operand strides bstride) write
// batches consecutive d x d outputs.
template <typename OutT>
bitsmoe_status run_symmetric(gemm::Problem p, int64_t d, double scale, OutT* out, void* stream,
                             const char* name, int64_t batches = 1) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int T = static_cast<int>((d + GT - 1) / GT);
  const int64_t ntiles = static_cast<int64_t>(T) * (T + 1) / 2;
  p.tiles_m = p.tiles_n = T;
  p.symmetric = 1;
  // Split-K.  The engine keeps one workgroup per CU, so the GEMM takes about
  // (rounds of workgroups over the CUs) x (K tiles per workgroup); each
  // split also writes a 256 x 256 fp32 partial tile that the reduction reads
  // back (about 0.14 K-tile times of the whole device per workgroup at HBM
  // speed).  The split minimizing the sum, with at least four K tiles per
  // workgroup.
  const int64_t kt = p.ktiles;  // in units of gemm::BK
  const int64_t cus = device_cus();
  const int64_t wg1 = ntiles * batches;
  int64_t splits = 1;
  double best = 0.0;
  for (int64_t sp = 1; sp <= std::max<int64_t>(1, kt / 4); ++sp) {
    const int64_t rounds = (wg1 * sp + cus - 1) / cus;
    const double cost = static_cast<double>(rounds * ((kt + sp - 1) / sp)) + 0.14 * wg1 * sp;
    if (sp == 1 || cost < best) {
      best = cost;
      splits = sp;
    }
  }
  p.splits = static_cast<int>(splits);
  if (batches > 65535) return fail(BITSMOE_ERR_SHAPE, std::string(name) + ": too many batches");
  bitsmoe_status st;
  const int64_t zstride = splits * ntiles * GT * GT;
  float* part = static_cast<float*>(
      scratch(kScratchPart, static_cast<size_t>(batches * zstride) * sizeof(float), stream, &st));
  if (!part) return st;
  PartialStore epi{part, ntiles, T, zstride};
  // one-dimensional XCD-aware grid: the tiles of one split (the same K slice
  // of the operands) run together on one XCD and share its L2
  if (ntiles * splits * batches > INT32_MAX)
    return fail(BITSMOE_ERR_SHAPE, std::string(name) + ": too many workgroups");
  p.flat = static_cast<int>(ntiles);
  dim3 grid(static_cast<unsigned>(ntiles * splits * batches), 1, 1);
  {
    KernelTimer timer(name, stream);
    hipLaunchKernelGGL((gemm::gemm_nt_kernel<GT, GT, 32, 4, PartialStore>), grid,
                       dim3(gemm::kThreads), 0, s, p, epi);
  }
  BITSMOE_LAUNCH_CHECK("gram: gemm launch");
  constexpr int NB = (GT / RB_ROWS) * (GT / RB_COLS);
  hipLaunchKernelGGL((sym_reduce_kernel<OutT>),
                     dim3(static_cast<unsigned>(ntiles * NB), static_cast<unsigned>(batches)),
                     dim3(256), 0, s, part, p.splits, ntiles, T, d, scale, out);
  BITSMOE_LAUNCH_CHECK("gram: reduce launch");
  return BITSMOE_OK;
}

}  // namespace
}  // namespace bitsmoe

using namespace bitsmoe;

namespace bitsmoe {
namespace {

// scale * R^T R for rows R [n][d] (bf16 or fp32): R is transposed into the
// K-tiled layout (K = rows, zero-padded to the engine's K alignment; fp32
// split into hi + lo) and multiplied by the symmetric split-K GEMM.
template <typename OutT>
bitsmoe_status gram_rows(const void* R_dev, bitsmoe_dtype rt, int64_t n, int64_t d, double scale,
                         OutT* out_dev, void* stream, const char* who) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t npad = (n + gemm::kKAlign - 1) / gemm::kKAlign * gemm::kKAlign;
  const bool f32 = rt == BITSMOE_F32;
  bitsmoe_status st;
  const int64_t d_pad = (d + GT - 1) / GT * GT;  // whole K-tiled row tiles
  uint16_t* hi = static_cast<uint16_t*>(scratch(kScratchA, d_pad * npad * 2, stream, &st));
  if (!hi) return st;
  uint16_t* lo = nullptr;
  if (f32) {
    lo = static_cast<uint16_t*>(scratch(kScratchB, d_pad * npad * 2, stream, &st));
    if (!lo) return st;
  }
  if ((npad + 63) / 64 > INT32_MAX) return fail(BITSMOE_ERR_SHAPE, std::string(who) + ": too many rows");
  dim3 tg(static_cast<unsigned>((npad + 63) / 64), static_cast<unsigned>((d + 63) / 64));
  if (f32)
    hipLaunchKernelGGL(transpose_split_kernel<true>, tg, dim3(256), 0, s, R_dev, n, d, npad, hi, lo);
  else
    hipLaunchKernelGGL(transpose_split_kernel<false>, tg, dim3(256), 0, s, R_dev, n, d, npad, hi, lo);
  BITSMOE_LAUNCH_CHECK(who);
  gemm::Problem p{};
  static_assert(BK == gemm::kTileK, "the K-tiled operands need the kernel's K step");
  p.a.rows = p.b.rows = d_pad;
  p.a.kstep = p.b.kstep = static_cast<int64_t>(GT) * gemm::kTileK;
  p.a.rtile = p.b.rtile = static_cast<int64_t>(GT) * npad;
  p.segs = 1;
  p.kseg = npad;
  if (f32) {
    p.passes = 3;  // hi*hi + hi*lo + lo*hi
    p.a.pass[0] = hi; p.b.pass[0] = hi;
    p.a.pass[1] = hi; p.b.pass[1] = lo;
    p.a.pass[2] = lo; p.b.pass[2] = hi;
  } else {
    p.passes = 1;
    p.a.pass[0] = p.b.pass[0] = hi;
  }
  p.ktiles = p.passes * npad / BK;
  return run_symmetric<OutT>(p, d, scale, out_dev, stream, who);
}

bitsmoe_status check_rows(const void* R_dev, const void* out_dev, bitsmoe_dtype rt, int64_t n,
                          int64_t d, const char* who) {
  if (!R_dev || !out_dev) return fail(BITSMOE_ERR_ARG, std::string(who) + ": null pointer");
  if (!aligned16({R_dev, out_dev}))
    return fail(BITSMOE_ERR_ARG, std::string(who) + ": device pointers must be 16-byte aligned");
  if (n <= 0 || d <= 0) return fail(BITSMOE_ERR_ARG, std::string(who) + ": non-positive size");
  if (rt != BITSMOE_F32 && rt != BITSMOE_BF16) return fail(BITSMOE_ERR_DTYPE, std::string(who) + ": dtype");
  if (d % 64 != 0) return fail(BITSMOE_ERR_SHAPE, std::string(who) + ": d must be a multiple of 64");
  return BITSMOE_OK;
}

}  // namespace
}  // namespace bitsmoe

extern "C" bitsmoe_status bitsmoe_gram(const void* X_dev, bitsmoe_dtype xt, int64_t n, int64_t d,
                                       float* H_dev, void* stream) {
  bitsmoe_status st = check_rows(X_dev, H_dev, xt, n, d, "gram");
  if (st != BITSMOE_OK) return st;
  st = gram_rows<float>(X_dev, xt, n, d, 1.0 / static_cast<double>(n), H_dev, stream, "gram");
  if (st != BITSMOE_OK) return st;
  return ok();
}

extern "C" bitsmoe_status bitsmoe_gram_experts_in(const void* W_dev, bitsmoe_dtype wt, int64_t E,
                                                  int64_t d_out, int64_t d_in, double* M_dev,
                                                  void* stream) {
  if (E <= 0 || d_out <= 0) return fail(BITSMOE_ERR_ARG, "gram_experts_in: non-positive size");
  if (d_out % 64 != 0)
    return fail(BITSMOE_ERR_SHAPE, "gram_experts_in: d_out and d_in must be multiples of 64");
  // the stacked expert rows W_cat = [W_1; ...; W_E] are [E * d_out][d_in]
  bitsmoe_status st = check_rows(W_dev, M_dev, wt, E * d_out, d_in, "gram_experts_in");
  if (st != BITSMOE_OK) return st;
  st = gram_rows<double>(W_dev, wt, E * d_out, d_in, 1.0, M_dev, stream, "gram_experts_in");
  if (st != BITSMOE_OK) return st;
  return ok();
}

extern "C" bitsmoe_status bitsmoe_gram_experts(const void* W_dev, bitsmoe_dtype wt, int64_t E,
                                               int64_t d_out, int64_t d_in, double* M_dev,
                                               void* stream) {
  if (!W_dev || !M_dev) return fail(BITSMOE_ERR_ARG, "gram_experts: null pointer");
  if (!aligned16({W_dev, M_dev}))
    return fail(BITSMOE_ERR_ARG, "gram_experts: device pointers must be 16-byte aligned");
  if (E <= 0 || d_out <= 0 || d_in <= 0) return fail(BITSMOE_ERR_ARG, "gram_experts: non-positive size");
  if (wt != BITSMOE_F32 && wt != BITSMOE_BF16) return fail(BITSMOE_ERR_DTYPE, "gram_experts: dtype");
  if (d_out % 64 != 0 || d_in % 64 != 0)
    return fail(BITSMOE_ERR_SHAPE, "gram_experts: d_out and d_in must be multiples of 64");
  hipStream_t s = static_cast<hipStream_t>(stream);
  gemm::Problem p{};
  p.a.ld = p.b.ld = d_in;
  p.a.estride = p.b.estride = d_out * d_in;
  p.a.rows = p.b.rows = d_out;
  p.segs = static_cast<int>(E);
  p.kseg = d_in;
  if (wt == BITSMOE_F32) {
    const int64_t count = E * d_out * d_in;
    bitsmoe_status st;
    uint16_t* hi = static_cast<uint16_t*>(scratch(kScratchA, count * 2, stream, &st));
    if (!hi) return st;
    uint16_t* lo = static_cast<uint16_t*>(scratch(kScratchB, count * 2, stream, &st));
    if (!lo) return st;
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 65536));
    hipLaunchKernelGGL(split_kernel, dim3(blocks), dim3(256), 0, s,
                       static_cast<const float*>(W_dev), count, hi, lo);
    BITSMOE_LAUNCH_CHECK("gram_experts: split launch");
    p.passes = 3;
    p.a.pass[0] = hi; p.b.pass[0] = hi;
    p.a.pass[1] = hi; p.b.pass[1] = lo;
    p.a.pass[2] = lo; p.b.pass[2] = hi;
  } else {
    p.passes = 1;
    p.a.pass[0] = p.b.pass[0] = static_cast<const uint16_t*>(W_dev);
  }
  p.ktiles = static_cast<int64_t>(p.passes) * E * d_in / BK;
  bitsmoe_status st = run_symmetric<double>(p, d_out, 1.0, M_dev, stream, "gram_experts");
  if (st != BITSMOE_OK) return st;
  return ok();
}

extern "C" bitsmoe_status bitsmoe_gram_routed(const void* X_dev, bitsmoe_dtype xt, int64_t n,
                                              int64_t d, int64_t E, const int64_t* offsets_host,
                                              const int32_t* rows_host, const float* weights_host,
                                              float* H_dev, void* stream) {
  bitsmoe_status st = check_rows(X_dev, H_dev, xt, n, d, "gram_routed");
  if (st != BITSMOE_OK) return st;
  if (!offsets_host || !rows_host || !weights_host)
    return fail(BITSMOE_ERR_ARG, "gram_routed: null pointer");
  if (E <= 0 || E > 65535) return fail(BITSMOE_ERR_ARG, "gram_routed: experts outside 1..65535");
  if (offsets_host[0] != 0) return fail(BITSMOE_ERR_ARG, "gram_routed: offsets[0] must be 0");
  int64_t nmax = 0;
  for (int64_t e = 0; e < E; ++e) {
    const int64_t c = offsets_host[e + 1] - offsets_host[e];
    if (c < 0) return fail(BITSMOE_ERR_ARG, "gram_routed: offsets must not decrease");
    nmax = std::max(nmax, c);
  }
  const int64_t total = offsets_host[E];
  for (int64_t i = 0; i < total; ++i) {
    if (rows_host[i] < 0 || rows_host[i] >= n)
      return fail(BITSMOE_ERR_ARG, "gram_routed: row index outside [0, n)");
    if (!(weights_host[i] >= 0.0f) || !std::isfinite(weights_host[i]))
      return fail(BITSMOE_ERR_ARG, "gram_routed: weights must be finite and non-negative");
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool f32 = xt == BITSMOE_F32;
  const int64_t npad = std::max<int64_t>(gemm::kKAlign,
                                         (nmax + gemm::kKAlign - 1) / gemm::kKAlign * gemm::kKAlign);
  const int64_t d_pad = (d + GT - 1) / GT * GT;
  const int64_t per = d_pad * npad;  // elements per expert and operand
  // routing tables on the device: offsets [E+1], rows [total], weights [total]
  const size_t tbytes = static_cast<size_t>(E + 1) * 8 + static_cast<size_t>(total) * 8 + 16;
  char* tab = static_cast<char*>(scratch(kScratchMisc, tbytes, stream, &st));
  if (!tab) return st;
  int64_t* off_d = reinterpret_cast<int64_t*>(tab);
  int32_t* rows_d = reinterpret_cast<int32_t*>(off_d + E + 1);
  float* w_d = reinterpret_cast<float*>(rows_d + total + (total & 1));
  hipError_t he = hipMemcpyAsync(off_d, offsets_host, (E + 1) * 8, hipMemcpyHostToDevice, s);
  if (he == hipSuccess && total > 0)
    he = hipMemcpyAsync(rows_d, rows_host, total * 4, hipMemcpyHostToDevice, s);
  if (he == hipSuccess && total > 0)
    he = hipMemcpyAsync(w_d, weights_host, total * 4, hipMemcpyHostToDevice, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);  // the host tables may go away after return
  if (he != hipSuccess) return device_error("gram_routed: routing table copy", he);
  uint16_t* A = static_cast<uint16_t*>(scratch(kScratchA, (f32 ? 2 : 1) * E * per * 2, stream, &st));
  if (!A) return st;
  uint16_t* B = static_cast<uint16_t*>(scratch(kScratchB, 2 * E * per * 2, stream, &st));
  if (!B) return st;
  uint16_t* a_lo = f32 ? A + E * per : nullptr;
  uint16_t* b_lo = B + E * per;
  dim3 tg(static_cast<unsigned>(npad / 64), static_cast<unsigned>((d + 63) / 64),
          static_cast<unsigned>(E));
  if (f32)
    hipLaunchKernelGGL(routed_gather_kernel<true>, tg, dim3(256), 0, s, X_dev, d, off_d, rows_d, w_d,
                       npad, d_pad, A, a_lo, B, b_lo);
  else
    hipLaunchKernelGGL(routed_gather_kernel<false>, tg, dim3(256), 0, s, X_dev, d, off_d, rows_d,
                       w_d, npad, d_pad, A, a_lo, B, b_lo);
  BITSMOE_LAUNCH_CHECK("gram_routed: gather launch");
  gemm::Problem p{};
  p.a.rows = p.b.rows = d_pad;
  p.a.kstep = p.b.kstep = static_cast<int64_t>(GT) * gemm::kTileK;
  p.a.rtile = p.b.rtile = static_cast<int64_t>(GT) * npad;
  p.a.bstride = p.b.bstride = per;
  p.segs = 1;
  p.kseg = npad;
  if (f32) {
    p.passes = 3;  // x_hi (wx)_hi + x_hi (wx)_lo + x_lo (wx)_hi
    p.a.pass[0] = A;    p.b.pass[0] = B;
    p.a.pass[1] = A;    p.b.pass[1] = b_lo;
    p.a.pass[2] = a_lo; p.b.pass[2] = B;
  } else {
    p.passes = 2;  // x (wx)_hi + x (wx)_lo, x exact in bf16
    p.a.pass[0] = A; p.b.pass[0] = B;
    p.a.pass[1] = A; p.b.pass[1] = b_lo;
  }
  p.ktiles = p.passes * npad / BK;
  st = run_symmetric<float>(p, d, 1.0 / static_cast<double>(n), H_dev, stream, "gram_routed", E);
  if (st != BITSMOE_OK) return st;
  return ok();
}
