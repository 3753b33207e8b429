// bf16 matrix-core ("NT") GEMM engine for gfx950.
//
// Every contraction of the quantizer has the form
//     acc[i][j] = sum_k A[i][k] * B[j][k]
// with both operands stored as bf16 rows that are contiguous along k: the
// calibration Gram (A = B = X^T), the cross-expert Gram (A = B = the expert
// rows, k running over experts and input channels), the spectral factors
// (A = U^T, B = W_e^T) and the loss table (A = off-diagonal H, B = error
// rows).  The engine takes a workgroup tile of BM x BN outputs, 4 waves of
// 64 lanes, stages K in steps of 32 through double-buffered LDS and issues
// v_mfma_f32_32x32x16_bf16.  What happens to the fp32 accumulators is left to
// an epilogue functor.
//
// The K index is a flattened (pass, segment, k) triple:
//   * passes   let one launch add up to 4 products A_p B_p^T into the same
//              accumulators (used for hi/lo bf16 splits of fp32 data);
//   * segments let K run over several equally long pieces that are a fixed
//              stride apart in memory (the experts of W for M = sum W_e W_e^T).
// gridDim.y splits K (split-K); gridDim.z is a batch index with its own
// operand strides.
#pragma once

#include "common.hpp"

namespace bitsmoe {
namespace gemm {

constexpr int BK = 32;             // K elements per LDS stage
constexpr int LDK = BK + 8;        // padded LDS row (80 bytes: conflict-free 16-byte reads)
constexpr int kThreads = 256;

struct Side {
  const uint16_t* pass[4];  // base pointer of each pass
  int64_t ld;               // elements between consecutive rows
  int64_t estride;          // elements between consecutive K segments
  int64_t bstride;          // elements between batches (blockIdx.z)
  int64_t rows;             // valid rows (rows beyond are read as zero)
};

struct Problem {
  Side a, b;
  int passes;
  int segs;          // K segments per pass
  int64_t kseg;      // K elements per segment (multiple of BK)
  int64_t ktiles;    // passes * segs * kseg / BK
  int splits;        // gridDim.y
  int tiles_m, tiles_n;
  int symmetric;     // 1: only tiles with tm <= tn are launched (gridDim.x = T(T+1)/2)
};

__device__ __forceinline__ void tile_coords(const Problem& p, int t, int* tm, int* tn) {
  if (!p.symmetric) {
    *tm = t / p.tiles_n;
    *tn = t % p.tiles_n;
    return;
  }
  int r = 0;
  while (t >= p.tiles_m - r) {
    t -= p.tiles_m - r;
    ++r;
  }
  *tm = r;
  *tn = r + t;
}

__device__ __forceinline__ const uint16_t* pass_ptr(const Side& s, int pass) {
  switch (pass) {
    case 0: return s.pass[0];
    case 1: return s.pass[1];
    case 2: return s.pass[2];
    default: return s.pass[3];
  }
}

// Address of element (row, k0) of K tile `kt` for operand side `s`.
__device__ __forceinline__ const uint16_t* tile_ptr(const Problem& p, const Side& s, int64_t kt,
                                                    int64_t row, int64_t z) {
  const int64_t tiles_seg = p.kseg / BK;
  const int64_t per_pass = static_cast<int64_t>(p.segs) * tiles_seg;
  const int pass = static_cast<int>(kt / per_pass);
  const int64_t rem = kt - static_cast<int64_t>(pass) * per_pass;
  const int64_t seg = rem / tiles_seg;
  const int64_t k0 = (rem - seg * tiles_seg) * BK;
  return pass_ptr(s, pass) + z * s.bstride + seg * s.estride + row * s.ld + k0;
}

// Accumulator fragment bookkeeping handed to epilogues.
template <int BM, int BN, int WM, int WN>
struct Frag {
  static constexpr int FM = BM / WM / 32;
  static constexpr int FN = BN / WN / 32;
  f32x16 acc[FM][FN];
  int tm, tn;        // tile coordinates
  int row0, col0;    // first row / column of this wave's sub-tile (global)
  int lane;
  int wm, wn, wave;
  int ks;            // split index
  int64_t z;         // batch index
  // global row of accumulator register r of fragment mi
  __device__ __forceinline__ int row(int mi, int r) const {
    return row0 + 32 * mi + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
  __device__ __forceinline__ int col(int ni) const { return col0 + 32 * ni + (lane & 31); }
};

template <int BM, int BN, int WM, int WN, class Epi>
__global__ __launch_bounds__(kThreads) void gemm_nt_kernel(Problem p, Epi epi) {
  static_assert(WM * WN == 4, "four waves");
  static_assert(BM % (32 * WM) == 0 && BN % (32 * WN) == 0, "wave tile");
  constexpr int ACH = BM * BK / 8 / kThreads;  // 16-byte chunks per thread
  constexpr int BCH = BN * BK / 8 / kThreads;
  static_assert(ACH >= 1 && BCH >= 1, "tile too small");
  using F = Frag<BM, BN, WM, WN>;

  __shared__ __align__(16) uint16_t As[2][BM * LDK];
  __shared__ __align__(16) uint16_t Bs[2][BN * LDK];

  const int tid = threadIdx.x;
  F f;
  f.lane = tid & 63;
  f.wave = tid >> 6;
  f.wm = f.wave / WN;
  f.wn = f.wave % WN;
  tile_coords(p, blockIdx.x, &f.tm, &f.tn);
  f.ks = blockIdx.y;
  f.z = blockIdx.z;
  f.row0 = f.tm * BM + f.wm * (BM / WM);
  f.col0 = f.tn * BN + f.wn * (BN / WN);
#pragma unroll
  for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
    for (int ni = 0; ni < F::FN; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) f.acc[mi][ni][r] = 0.0f;

  const int64_t kt0 = p.ktiles * f.ks / p.splits;
  const int64_t kt1 = p.ktiles * (f.ks + 1) / p.splits;

  uint4 ra[ACH], rb[BCH];
  auto load = [&](int64_t kt) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + kThreads * i;
      const int r = c >> 2, k8 = (c & 3) * 8;
      const int64_t gr = static_cast<int64_t>(f.tm) * BM + r;
      ra[i] = (gr < p.a.rows) ? *reinterpret_cast<const uint4*>(tile_ptr(p, p.a, kt, gr, f.z) + k8)
                              : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + kThreads * i;
      const int r = c >> 2, k8 = (c & 3) * 8;
      const int64_t gr = static_cast<int64_t>(f.tn) * BN + r;
      rb[i] = (gr < p.b.rows) ? *reinterpret_cast<const uint4*>(tile_ptr(p, p.b, kt, gr, f.z) + k8)
                              : make_uint4(0, 0, 0, 0);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + kThreads * i;
      *reinterpret_cast<uint4*>(&As[buf][(c >> 2) * LDK + (c & 3) * 8]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + kThreads * i;
      *reinterpret_cast<uint4*>(&Bs[buf][(c >> 2) * LDK + (c & 3) * 8]) = rb[i];
    }
  };

  if (kt0 < kt1) {
    load(kt0);
    store(0);
    __syncthreads();
    int buf = 0;
    const int arow = f.wm * (BM / WM) + (f.lane & 31);
    const int brow = f.wn * (BN / WN) + (f.lane & 31);
    const int kq = 8 * (f.lane >> 5);
    for (int64_t kt = kt0; kt < kt1; ++kt) {
      const bool more = kt + 1 < kt1;
      if (more) load(kt + 1);
#pragma unroll
      for (int kk = 0; kk < BK; kk += 16) {
        bf16x8 af[F::FM], bfr[F::FN];
#pragma unroll
        for (int mi = 0; mi < F::FM; ++mi)
          af[mi] = *reinterpret_cast<const bf16x8*>(&As[buf][(arow + 32 * mi) * LDK + kk + kq]);
#pragma unroll
        for (int ni = 0; ni < F::FN; ++ni)
          bfr[ni] = *reinterpret_cast<const bf16x8*>(&Bs[buf][(brow + 32 * ni) * LDK + kk + kq]);
#pragma unroll
        for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
          for (int ni = 0; ni < F::FN; ++ni)
            f.acc[mi][ni] =
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bfr[ni], f.acc[mi][ni], 0, 0, 0);
      }
      if (more) store(buf ^ 1);
      __syncthreads();
      buf ^= 1;
    }
  }
  epi(f);
}

}  // namespace gemm
}  // namespace bitsmoe
