// Stage 3: serve one projection of an MoE layer from its packed factors.
//
// The paper dequantizes the packed expert-specific factors inside the expert
// kernels (Sec. 4.4).  With the output-space basis an expert is
// W_e ~ U C^_e, so a token x routed to experts e_j with weights g_j gives
//     y = U z,   z = sum_j g_j C^_{e_j} x,
// the shared basis applied once per token whatever the number of routed
// experts.
//   1. decode_z_kernel  a job is (expert, up to T of its routing entries);
//                       each lane owns 32-entry segments of a unit row (one
//                       32-bit word of every bit plane, one group parameter)
//                       and holds the jobs' token values of its segment in
//                       registers across the rows its wave walks:
//                       zp[i][k] = w_i (c^_{e,k} . x_{tok_i}).
//   2. decode_y_kernel  per token tile: z = sum of each token's partials
//                       (fixed order) staged in LDS, y = U z with 16 waves
//                       splitting r and one lane per output column.
//
// Decoding a segment: entry j of the segment is bit j of each plane word, so
// four entries at a time the planes' nibbles are spread to one byte per
// entry (nibble * 0x204081 places bit i at bit 8i with no carries) and
// or-ed, plane t shifted by t; the bytes convert to floats exactly.  The
// group's affine step is applied once per segment:
//     sum_j (q_j s + m) x_j = s sum_j q_j x_j + m sum_j x_j.
#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "bitsmoe.h"
#include "common.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

constexpr int kWaves = 4;      // waves per decode_z workgroup
constexpr int kSeg = 32;       // entries per lane segment
constexpr int kYWaves = 16;    // waves per decode_y workgroup

__device__ __forceinline__ bool width_ok(int b) {
  return b == 0 || b == 16 || (b >= 1 && b <= BITSMOE_MAX_BITS);
}

// s_waitcnt vmcnt(0) alone (expcnt and lgkmcnt left at their maxima), in
// the gfx9 encoding.
__device__ __forceinline__ void wait_vmcnt0() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// bits 0..3 of v -> bit 0 of bytes 0..3
__device__ __forceinline__ uint32_t spread4(uint32_t v) {
  return __umul24(v & 15u, 0x204081u) & 0x01010101u;
}
// nibble n (< 16) -> its bits at bit t of bytes 0..3.  The shift goes into
// the multiplier while that stays within 24 bits (a full-rate v_mul_u32_u24);
// past that the nibble is shifted first.
__device__ __forceinline__ uint32_t spread4_at(uint32_t n, int t) {
  return t <= 2 ? __umul24(n, 0x204081u << t) & (0x01010101u << t)
                : __umul24(n << t, 0x204081u) & (0x01010101u << t);
}

// A row's packed state as one lane sees it: width (0 when the unit is
// evicted or inconsistent), first word, its segment's plane words and group
// parameter.
struct RowFetch {
  int b;
  int64_t o0;
  uint32_t pw[BITSMOE_MAX_BITS];
  uint32_t prm;
};

// One job per blockIdx.y: jobs[2j] = {expert, first routing entry, entries
// (1..T), 0}, jobs[2j+1] = the entries' tokens.  Each wave walks `passes`
// passes of R = 64 / L rows (L lanes per row, a power of two); a row of
// nseg = d / 32 segments takes ceil(nseg / L) slices.  ONE_SLICE
// (nseg <= L) keeps the token values in registers for all the wave's rows
// and fetches the next row's plane words while the current one is summed.
// The row descriptors (width, offsets) of the wave's rows are loaded once,
// lane sub * L + p holding pass p of row group sub (passes <= L).
// TOPK (T = 1): job j is routing slot j of a [B][kk] top-k table instead,
// expert topk[j], token j / kk, weight ew[j]; an expert outside [0, E)
// gives a zero partial.
template <int T, bool ONE_SLICE, bool TOPK>
__global__ __launch_bounds__(256) void decode_z_kernel(
    const uint32_t* __restrict__ codes32, const uint32_t* __restrict__ params,
    const uint8_t* __restrict__ bits, const int64_t* __restrict__ off, int64_t total_words,
    int r, int d, int G, int L, int passes, const float* __restrict__ X,
    const int4* __restrict__ jobs, const int32_t* __restrict__ topk, int kk, int E,
    const float* __restrict__ ew, float* __restrict__ zp) {
  static_assert(!TOPK || T == 1, "top-k jobs hold one routing entry");
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int e, nt;
  int64_t i0;
  int4 jt;
  bool dead = false;
  if (TOPK) {
    e = topk[blockIdx.y];
    dead = e < 0 || e >= E;
    if (dead) e = 0;
    i0 = blockIdx.y;
    nt = 1;
    jt = make_int4(static_cast<int>(blockIdx.y) / kk, 0, 0, 0);
  } else {
    const int4 job = jobs[2 * blockIdx.y];
    jt = jobs[2 * blockIdx.y + 1];
    e = job.x;
    i0 = job.y;
    nt = job.z;
  }
  const int R = 64 / L;
  const int sub = lane / L, sl = lane % L;
  const int nseg = d / kSeg;
  const int ns = (nseg + L - 1) / L;
  const int64_t nw = d / 64;
  const int kbase = (static_cast<int>(blockIdx.x) * kWaves + wave) * passes * R;
  if (kbase >= r) return;  // whole wave
  // row descriptors
  int db = 0;
  int64_t do0 = 0;
  {
    const int k = kbase + sl * R + sub;
    if (sl < passes && k < r) {
      const int64_t u = static_cast<int64_t>(e) * r + k;
      const int b = bits[u];
      const int64_t o0 = off[u], o1 = off[u + 1];
      // a unit whose width or offsets are inconsistent contributes nothing
      // (as bitsmoe_pack leaves it unwritten); width 0 is evicted
      const bool valid = width_ok(b) && b != 0 && o1 - o0 == b * nw && o0 >= 0 && o1 <= total_words;
      db = valid && !dead ? b : 0;
      do0 = valid && !dead ? o0 : 0;
    }
  }
  const int tk[4] = {jt.x, jt.y, jt.z, jt.w};
  const float* xrow[T];
#pragma unroll
  for (int t = 0; t < T; ++t) xrow[t] = X + static_cast<int64_t>(tk[t < nt ? t : 0]) * d;
  float x[T][kSeg], xs[T];
  auto load_x = [&](int seg) {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      xs[t] = 0.0f;
      if (t < nt && seg < nseg) {
        const float4* p4 = reinterpret_cast<const float4*>(xrow[t] + seg * kSeg);
#pragma unroll
        for (int q = 0; q < kSeg / 4; ++q) {
          const float4 v = p4[q];
          x[t][4 * q] = v.x;
          x[t][4 * q + 1] = v.y;
          x[t][4 * q + 2] = v.z;
          x[t][4 * q + 3] = v.w;
        }
#pragma unroll
        for (int j = 0; j < kSeg; ++j) xs[t] += x[t][j];
      } else {
#pragma unroll
        for (int j = 0; j < kSeg; ++j) x[t][j] = 0.0f;
      }
    }
  };
  // the descriptor of pass p for this lane's row group
  auto row_of = [&](int p, RowFetch& f) {
    const int src = sub * L + p;
    f.b = __shfl(db, src, 64);
    const int lo = __shfl(static_cast<int>(do0 & 0xffffffff), src, 64);
    const int hi = __shfl(static_cast<int>(do0 >> 32), src, 64);
    f.o0 = (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
  };
  // plane words and parameter of segment seg (widths 1..8)
  auto fetch_planes = [&](int k, int seg, RowFetch& f) {
    if (f.b >= 1 && f.b <= BITSMOE_MAX_BITS && seg < nseg && k < r) {
      const int64_t u = static_cast<int64_t>(e) * r + k;
      const uint32_t* pw = codes32 + 2 * f.o0 + seg;
#pragma unroll
      for (int t = 0; t < BITSMOE_MAX_BITS; ++t)
        if (t < f.b) f.pw[t] = pw[2 * t * nw];
      f.prm = params[u * (d / G) + (seg * kSeg) / G];
    }
  };
  // sum over the segment: acc[t] += sum_j c^_j x[t][j]
  auto seg_dot = [&](const RowFetch& f, int seg, float (&acc)[T]) {
    float dq[T];
#pragma unroll
    for (int t = 0; t < T; ++t) dq[t] = 0.0f;
    if (f.b == 16) {
      // fp16 row: entries 32 seg .. 32 seg + 31 at byte 8 o0 + 64 seg
      const uint2* h = reinterpret_cast<const uint2*>(codes32 + 2 * f.o0) + 8 * seg;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const uint2 v = h[q];
        const float c[4] = {f16_bits_to_f32(static_cast<uint16_t>(v.x & 0xffffu)),
                            f16_bits_to_f32(static_cast<uint16_t>(v.x >> 16)),
                            f16_bits_to_f32(static_cast<uint16_t>(v.y & 0xffffu)),
                            f16_bits_to_f32(static_cast<uint16_t>(v.y >> 16))};
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4)
#pragma unroll
          for (int t = 0; t < T; ++t) dq[t] = fmaf(c[c4], x[t][4 * q + c4], dq[t]);
      }
#pragma unroll
      for (int t = 0; t < T; ++t) acc[t] += dq[t];
      return;
    }
    const float s = f16_bits_to_f32(static_cast<uint16_t>(f.prm & 0xffffu));
    const float m = f16_bits_to_f32(static_cast<uint16_t>(f.prm >> 16));
    uint32_t qb[kSeg / 4];
#pragma unroll
    for (int kk = 0; kk < kSeg / 4; ++kk) qb[kk] = spread4(f.pw[0] >> (4 * kk));
#pragma unroll
    for (int t = 1; t < BITSMOE_MAX_BITS; ++t)
      if (t < f.b) {
#pragma unroll
        for (int kk = 0; kk < kSeg / 4; ++kk) qb[kk] |= spread4(f.pw[t] >> (4 * kk)) << t;
      }
#pragma unroll
    for (int kk = 0; kk < kSeg / 4; ++kk) {
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) {
        const float q = static_cast<float>((qb[kk] >> (8 * c4)) & 0xffu);
#pragma unroll
        for (int t = 0; t < T; ++t) dq[t] = fmaf(q, x[t][4 * kk + c4], dq[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < T; ++t) acc[t] += fmaf(s, dq[t], m * xs[t]);
  };
  auto finish_row = [&](int k, float (&acc)[T]) {
    // sum over the L lanes of each row (lane groups are aligned powers of two)
    for (int mlane = L / 2; mlane >= 1; mlane >>= 1)
#pragma unroll
      for (int t = 0; t < T; ++t) acc[t] += __shfl_xor(acc[t], mlane, 64);
    if (k < r && sl == 0) {
#pragma unroll
      for (int t = 0; t < T; ++t)
        if (t < nt) zp[(i0 + t) * r + k] = dead ? 0.0f : ew[i0 + t] * acc[t];
    }
  };
  if (ONE_SLICE) {
    load_x(sl);
    RowFetch cur, nxt;
    nxt.b = 0;
    nxt.o0 = 0;
    row_of(0, cur);
    fetch_planes(kbase + sub, sl, cur);
    for (int pass = 0; pass < passes; ++pass) {
      const int k = kbase + pass * R + sub;
      if (pass + 1 < passes) {
        row_of(pass + 1, nxt);
        fetch_planes(k + R, sl, nxt);
      }
      float acc[T];
#pragma unroll
      for (int t = 0; t < T; ++t) acc[t] = 0.0f;
      if (k < r && cur.b != 0 && sl < nseg) seg_dot(cur, sl, acc);
      finish_row(k, acc);
      cur = nxt;
    }
  } else {
    for (int pass = 0; pass < passes; ++pass) {
      const int k = kbase + pass * R + sub;
      RowFetch f;
      row_of(pass, f);
      float acc[T];
#pragma unroll
      for (int t = 0; t < T; ++t) acc[t] = 0.0f;
      if (k < r && f.b != 0) {
        for (int sidx = 0; sidx < ns; ++sidx) {
          const int seg = sidx * L + sl;
          load_x(seg);
          if (seg >= nseg) continue;
          fetch_planes(k, seg, f);
          seg_dot(f, seg, acc);
        }
      }
      finish_row(k, acc);
    }
  }
}

// y[b][o] = sum_k Ut[k][o] z_b[k], z_b[k] = sum over token b's routing
// entries (in the order given) of zp[i][k]: the entries pidx[b][0..kmax)
// (-1 = none), or b kmax .. b kmax + kmax - 1 when pidx is null.  TB tokens per workgroup
// (blockIdx.y), 64 output columns per workgroup (blockIdx.x); wave w takes
// the contiguous rows [w nk, (w + 1) nk) (nk a multiple of 4), fetching U
// 16 rows ahead, and the 16 partial sums are added in wave order.
template <int TB>
__global__ __launch_bounds__(1024) void decode_y_kernel(const float* __restrict__ zp,
                                                        const int64_t* __restrict__ pidx, int kmax,
                                                        int r, const float* __restrict__ Ut,
                                                        int64_t d_out, int64_t B,
                                                        float* __restrict__ Y) {
  constexpr int KC = 16;
  extern __shared__ float sm[];  // z [TB][rp], then partials [16][TB][64]
  const int nk = ((r + kYWaves - 1) / kYWaves + 3) / 4 * 4;
  const int rp = nk * kYWaves;  // r padded (z is 0 past r)
  float* z = sm;
  float* red = sm + TB * rp;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t o = static_cast<int64_t>(blockIdx.x) * 64 + lane;
  const int k0 = wave * nk;
  const bool col = o < d_out;
  float ua[KC], ub[KC];
  auto fetch = [&](int c, float (&u)[KC]) {
#pragma unroll
    for (int i = 0; i < KC; ++i) {
      const int k = k0 + c * KC + i;
      u[i] = (col && c * KC + i < nk && k < r) ? Ut[static_cast<int64_t>(k) * d_out + o] : 0.0f;
    }
  };
  fetch(0, ua);
  const int64_t b0 = static_cast<int64_t>(blockIdx.y) * TB;
  for (int idx = threadIdx.x; idx < TB * rp; idx += 64 * kYWaves) {
    const int tb = idx / rp, k = idx - tb * rp;
    const int64_t b = b0 + tb;
    float s = 0.0f;
    if (b < B && k < r) {
      for (int j = 0; j < kmax; ++j) {
        const int64_t i = pidx ? pidx[b * kmax + j] : b * kmax + j;
        if (i >= 0) s += zp[i * r + k];
      }
    }
    z[idx] = s;
  }
  __syncthreads();
  float acc[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) acc[tb] = 0.0f;
  const int nc = (nk + KC - 1) / KC;
  for (int c = 0; c < nc; ++c) {
    if (c + 1 < nc) fetch(c + 1, ub);
#pragma unroll
    for (int i4 = 0; i4 < KC / 4; ++i4) {
      const int kk = k0 + c * KC + 4 * i4;  // < rp: nk is a multiple of 4
      if (c * KC + 4 * i4 < nk) {
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          const float4 zv = *reinterpret_cast<const float4*>(z + tb * rp + kk);
          acc[tb] = fmaf(ua[4 * i4], zv.x, acc[tb]);
          acc[tb] = fmaf(ua[4 * i4 + 1], zv.y, acc[tb]);
          acc[tb] = fmaf(ua[4 * i4 + 2], zv.z, acc[tb]);
          acc[tb] = fmaf(ua[4 * i4 + 3], zv.w, acc[tb]);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < KC; ++i) ua[i] = ub[i];
  }
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) red[(wave * TB + tb) * 64 + lane] = acc[tb];
  __syncthreads();
  if (wave < TB) {
    const int tb = wave;
    float s = 0.0f;
    for (int w = 0; w < kYWaves; ++w) s += red[(w * TB + tb) * 64 + lane];
    const int64_t b = b0 + tb;
    if (b < B && o < d_out) Y[b * d_out + o] = s;
  }
}

// ---- batches: z and y on the matrix cores ----
//
// Each expert's routing entries are taken in jobs of up to 16 tokens and
// its unit rows in blocks of 16 (one wave each), so that
//     Z[t][k] = sum_g s_{k,g} sum_{i in g} q_{k,i} x_t[i] + m_{k,g} sum_{i in g} x_t[i]
// runs as v_mfma_f32_16x16x32_f16: A = the tokens' x as fp16 hi + lo (two
// products; x = hi + lo to about 2^-22), B = the codes q of 16 rows (small
// integers, exact in fp16), one fresh accumulator per group of G entries,
// scaled by s and shifted by m times the token's group sum in fp32.  An
// expert's codes are decoded once per job instead of once per routing
// entry.  The token sums of the partial rows then go through the shared
// basis as an fp32 matrix product (v_mfma_f32_16x16x4_f32).

constexpr int kMmaWaves = 4;    // waves per z workgroup (16 unit rows each)
constexpr int kMmaStages = 4;   // LDS ring of the z step: stages loaded 3 ahead

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));

// x [B][d] fp32 -> xh, xl [B][d] fp16 (x ~ xh + xl) and xs [B][d / G] fp32
// (the sum of each block of G entries; the z step passes min(group, 128)),
// for block index idx = token * (d / G) + block, by one wave: each lane
// converts up to four entries and the block sum is a wave reduction.
__device__ __forceinline__ void xprep_wave(const float* __restrict__ X, int64_t idx, int d, int G,
                                           _Float16* __restrict__ xh, _Float16* __restrict__ xl,
                                           float* __restrict__ xs) {
  const int ng = d / G;
  const int lane = threadIdx.x & 63;
  const int64_t b = idx / ng;
  const int g = static_cast<int>(idx - b * ng);
  const int64_t base = b * d + static_cast<int64_t>(g) * G;
  float sum = 0.0f;
  for (int i = 4 * lane; i < G; i += 256) {
    const float4 v = *reinterpret_cast<const float4*>(X + base + i);
    const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const _Float16 hh = static_cast<_Float16>(vv[j]);
      xh[base + i + j] = hh;
      xl[base + i + j] = static_cast<_Float16>(vv[j] - static_cast<float>(hh));
      sum += vv[j];
    }
  }
  sum = wave_sum(sum);
  if (lane == 0) xs[idx] = sum;
}

// Exclusive prefix sum over the 1024 threads of a workgroup (in thread
// order) of one int each; `sh` is 16 ints of LDS.  Returns the thread's
// exclusive sum and sets *total.
__device__ __forceinline__ int block_scan_1024(int v, int* sh, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(incl, o, 64);
    if (lane >= o) incl += u;
  }
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < 16; ++w) {
    const int t = sh[w];
    before += w < wave ? t : 0;
    all += t;
  }
  __syncthreads();  // sh may be reused by the caller
  *total = all;
  return before + incl - v;
}

// Groups a device top-k table [B][kk] by expert: jobs {expert, first sorted
// position, entries (1..jt), 0}, the number of jobs, and per sorted position
// the entry (b kk + j), its token and weight.  A slot whose expert is
// outside [0, E) has its partial row zp[entry][0..r) set to zero instead.
// The order of an expert's entries among its positions is not fixed
// (atomics), which changes nothing: each token's column of the product is
// computed on its own.  Workgroup 0 does the routing (when topk is set);
// the others, 16 waves each, run xprep_wave over the B (d / G) blocks.
constexpr int kRouteThreads = 1024;
constexpr int kRouteMaxExperts = 4096;  // four per thread in the scan
__global__ __launch_bounds__(kRouteThreads) void prep_kernel(
    const int32_t* __restrict__ topk, const float* __restrict__ topw, int64_t BK, int kk, int E,
    int r, int jt, int4* __restrict__ jobs, int* __restrict__ njobs, int32_t* __restrict__ ent,
    int32_t* __restrict__ tok, float* __restrict__ wgt, float* __restrict__ zp,
    const float* __restrict__ X, int64_t nblk, int d, int G, _Float16* __restrict__ xh,
    _Float16* __restrict__ xl, float* __restrict__ xs) {
  const int route = topk ? 1 : 0;
  if (static_cast<int>(blockIdx.x) >= route) {
    const int64_t idx = (static_cast<int64_t>(blockIdx.x) - route) * 16 + (threadIdx.x >> 6);
    if (idx < nblk) xprep_wave(X, idx, d, G, xh, xl, xs);
    return;
  }
  __shared__ int cnt[kRouteMaxExperts];
  __shared__ int start[kRouteMaxExperts];
  __shared__ int jstart[kRouteMaxExperts];
  __shared__ int sh[16];
  for (int e = threadIdx.x; e < E; e += kRouteThreads) cnt[e] = 0;
  __syncthreads();
  for (int64_t i = threadIdx.x; i < BK; i += kRouteThreads) {
    const int e = topk[i];
    if (e >= 0 && e < E) {
      atomicAdd(&cnt[e], 1);
    } else {
      for (int k = 0; k < r; ++k) zp[i * r + k] = 0.0f;
    }
  }
  __syncthreads();
  // positions and jobs: thread t owns experts 4t .. 4t + 3
  int c4[4], n4 = 0, j4 = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = 4 * static_cast<int>(threadIdx.x) + u;
    c4[u] = e < E ? cnt[e] : 0;
    n4 += c4[u];
    j4 += (c4[u] + jt - 1) / jt;
  }
  int ntot, jtot;
  int pos = block_scan_1024(n4, sh, &ntot);
  int jb = block_scan_1024(j4, sh, &jtot);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = 4 * static_cast<int>(threadIdx.x) + u;
    if (e < E) {
      start[e] = pos;
      jstart[e] = jb;
      for (int j = 0; j * jt < c4[u]; ++j)
        jobs[jb + j] = make_int4(e, pos + j * jt, min(jt, c4[u] - j * jt), 0);
      cnt[e] = 0;  // reused as the fill count below
    }
    pos += c4[u];
    jb += (c4[u] + jt - 1) / jt;
  }
  if (threadIdx.x == 0) *njobs = jtot;
  __syncthreads();
  for (int64_t i = threadIdx.x; i < BK; i += kRouteThreads) {
    const int e = topk[i];
    if (e >= 0 && e < E) {
      const int p = start[e] + atomicAdd(&cnt[e], 1);
      ent[p] = static_cast<int32_t>(i);
      tok[p] = static_cast<int32_t>(i / kk);
      wgt[p] = topw[i];
    }
  }
}

// The fp16 codes of 8 consecutive entries from their bit planes: bits
// sh .. sh + 7 of plane word w[t] are bit t of the 8 codes (entry j at bit
// sh + j; words of planes the row does not have are zero).  Each nibble's
// bits are spread to one byte per entry, and byte q becomes the fp16 of
// 1024 + q (0x6400 | q), minus 1024: exact.  Planes from bw on are skipped;
// bw is the same in every lane of the wave, so that the loop has no
// divergent branch.
__device__ __forceinline__ half8 codes8(const uint32_t (&w)[BITSMOE_MAX_BITS], int sh, int bw) {
  uint32_t qlo = 0, qhi = 0;
#pragma unroll
  for (int t = 0; t < BITSMOE_MAX_BITS; ++t) {
    if (t < bw) {
      qlo |= spread4_at((w[t] >> sh) & 15u, t);
      qhi |= spread4_at((w[t] >> (sh + 4)) & 15u, t);
    }
  }
  // bytes 2i, 2i + 1 of q and 0x64 above each: v_perm_b32 selector bytes 0-3
  // pick q, 4 picks 0x64
  const uint32_t hi8 = 0x64646464u;
  const uint32_t h[4] = {__builtin_amdgcn_perm(hi8, qlo, 0x04010400u),
                         __builtin_amdgcn_perm(hi8, qlo, 0x04030402u),
                         __builtin_amdgcn_perm(hi8, qhi, 0x04010400u),
                         __builtin_amdgcn_perm(hi8, qhi, 0x04030402u)};
  const half8 k1024 = {1024, 1024, 1024, 1024, 1024, 1024, 1024, 1024};
  return __builtin_bit_cast(half8, h) - k1024;
}

// One wave-wide direct global->LDS load: lane l reads 16 (4) bytes at its
// own address g and they land at LDS byte address lds + 16 l (+ 4 l); `lds`
// is wave-uniform.  Issued through inline assembly so that the compiler
// neither tracks the load nor inserts waits for it: the caller waits with
// s_waitcnt vmcnt and synchronizes the workgroup before reading.  M0 carries
// the LDS address; nothing else in the kernel uses M0.
__device__ __forceinline__ void lds_dma16(const void* g, const void* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds)));
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(g), "s"(l) : "memory");
}
__device__ __forceinline__ void lds_dma4(const void* g, const void* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds)));
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" : : "v"(g), "s"(l) : "memory");
}
// s_waitcnt vmcnt(N) alone, in the gfx9 encoding (vmcnt[3:0] in bits 3:0,
// vmcnt[5:4] in bits 15:14).
template <int N>
__device__ __forceinline__ void wait_vmcnt_n() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// zp[ent[p]][k] = wgt[p] (c^_{e,k} . x_{tok[p]}) for the positions p of job
// blockIdx.y (jobs[j] = {e, first, n <= TS, 0}; ent null: the position is
// the entry) and the 16 WV unit rows of block blockIdx.x, 16 per wave, as
// v_mfma_f32_16x16x32_f16 with the job's tokens as A (M; rows past TS are
// zero) and the codes as B (N): lane l holds row l % 16 and, of every
// 32-entry step, the 8 entries of chunk l / 16, and ends with the sums of
// that row for tokens 4 (l / 16) + i.
//
// The entries go by stages of 128 (four steps).  Within a stage a group (or
// the stage's half of a 256-entry group: a sub-group of GB = min(G, 128)
// entries) is dealt to its steps so that chunk c is GB / 4 consecutive
// entries; the stage's bits of a row's bit plane are 16 bytes, and chunk c of
// a step is one byte of them.  Every stage is fetched straight into LDS by
// the workgroup NS - 1 stages ahead (a ring of NS buffers): the tokens' x
// (fp16 hi and lo, in the order the lanes read them), their sub-group sums,
// and per wave the 16 rows' planes 0..3 and parameter words.  Every lane
// issues every load of a stage (a lane without a row or token reads a valid
// stand-in whose value goes unused, and the tail reloads the last stage), so
// a wave has a fixed number of loads per stage and the wait before a stage
// is exact.  Rows of 5 to 8 bits load their planes 4 and up, and fp16 rows
// their values, when the stage is summed.  With njobs set, jobs at or past
// *njobs return at once (the grid covers a bound).
constexpr int kRingPlanes = 4;  // bit planes fetched ahead

template <int G, int TS, int WV, int NS>
__global__ __launch_bounds__(64 * WV) void decode_zmma_kernel(
    const uint32_t* __restrict__ codes32, const uint32_t* __restrict__ params,
    const uint8_t* __restrict__ bits, const int64_t* __restrict__ off, int64_t total_words, int r,
    int d, const _Float16* __restrict__ xh, const _Float16* __restrict__ xl,
    const float* __restrict__ xs, const int4* __restrict__ jobs, const int* __restrict__ njobs,
    const int32_t* __restrict__ ent, const int32_t* __restrict__ tok,
    const float* __restrict__ wgt, float* __restrict__ zp) {
  constexpr int GB = G < 128 ? G : 128;  // sub-group: the part of a group within a stage
  constexpr int SG = GB / 32;            // MFMA steps per sub-group
  constexpr int NSUB = 128 / GB;         // sub-groups per stage
  constexpr int CH = GB / 4;             // entries of a sub-group per chunk
  constexpr int XSLOT = 16 * TS;         // 16-byte x slots of a stage (hi; lo alike)
  constexpr int XI = 2 * XSLOT / 64;     // x loads per stage (64 lanes each)
  constexpr int XPW = XI > WV ? XI / WV : 1;  // x loads per wave (waves past XI repeat one)
  constexpr int PER = XPW + 3;           // loads per wave per stage: x, planes, params, sums
  constexpr int RP = kRingPlanes;
  static_assert(XI % WV == 0 || WV % XI == 0, "x loads spread evenly over the waves");
  static_assert((NS - 2) * PER < 64, "vmcnt holds at most 63 loads");
  struct Stage {
    uint4 x[2][XSLOT];          // [hi, lo][(step * 4 + chunk) * TS + token]
    uint4 w[WV][RP][16];        // [wave][plane][row]: the row's 128 bits of the stage
    uint32_t prm[WV][4][16];    // [wave][sub-group][row]
    float4 sum[4][4];           // [sub-group][token / 4]
  };
  __shared__ Stage st[NS];
  if (njobs && static_cast<int>(blockIdx.y) >= *njobs) return;  // whole workgroup
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int4 jb = jobs[blockIdx.y];
  const int e = jb.x, first = jb.y, n = jb.z;
  const int64_t nw = d / 64;
  const int ng = d / G;
  const int nsb = d / GB;    // sub-groups of a unit row
  const int nst = d / 128;   // stages

  // this lane's unit row (lane % 16 of the wave's 16) and its width (0:
  // evicted, inconsistent or past r)
  const int rho = lane & 15, c = lane >> 4;
  const int k = static_cast<int>(blockIdx.x) * (16 * WV) + 16 * wave + rho;
  int ba = 0;
  int64_t oa = 0;
  if (k < r) {
    const int64_t u = static_cast<int64_t>(e) * r + k;
    const int b = bits[u];
    const int64_t o0 = off[u], o1 = off[u + 1];
    const bool valid = width_ok(b) && b != 0 && o1 - o0 == b * nw && o0 >= 0 && o1 <= total_words;
    ba = valid ? b : 0;
    oa = valid ? o0 : 0;
  }
  const bool packed = ba >= 1 && ba <= BITSMOE_MAX_BITS;
  const uint32_t* pw = codes32 + 2 * oa;  // plane t starts at word 2 t nw
  const void* standin = xh;               // a valid address for unused lanes

  // load addresses of this lane, all but the stage offset
  // x: slot xs0 + lane of load m = wave + WV i, part m / (XI / 2)
  const _Float16* xsrc[XPW];
#pragma unroll
  for (int i = 0; i < XPW; ++i) {
    const int m = (wave + WV * i) % XI;
    const int part = m / (XI / 2);
    const int slot = (m % (XI / 2)) * 64 + lane;
    const int tt = slot % TS, cc = (slot / TS) % 4, q = slot / (4 * TS);
    const int sg = q / SG, qq = q % SG;
    const int tk = tok[first + min(tt, n - 1)];
    xsrc[i] = (part ? xl : xh) + static_cast<int64_t>(tk) * d + sg * GB + cc * CH + 8 * qq;
  }
  // sums: sub-group c (lane / 16) of token rho, stand-in past NSUB or n
  const float* ssrc;
  {
    const int tk = tok[first + min(rho, n - 1)];
    ssrc = c < NSUB ? xs + static_cast<int64_t>(tk) * nsb + c : static_cast<const float*>(standin);
  }
  // planes: plane c of row rho (the 64 lanes cover 16 rows x 4 planes)
  const uint32_t* wsrc = (packed && c < min(ba, RP)) ? pw + 2 * c * nw
                                                     : static_cast<const uint32_t*>(standin);
  // parameters: sub-group c of row rho
  const uint32_t* psrc = (packed && c < NSUB)
                             ? params + (static_cast<int64_t>(e) * r + k) * ng
                             : static_cast<const uint32_t*>(standin);
  auto issue = [&](int s, int buf) {
    s = min(s, nst - 1);
    Stage& S = st[buf];
#pragma unroll
    for (int i = 0; i < XPW; ++i) {
      const int m = (wave + WV * i) % XI;
      lds_dma16(xsrc[i] + 128 * static_cast<int64_t>(s),
                &S.x[m / (XI / 2)][(m % (XI / 2)) * 64]);
    }
    lds_dma16(wsrc == standin ? wsrc : wsrc + 4 * s, &S.w[wave][0][0]);
    // the parameter word of sub-group c of stage s: group (128 s + GB c) / G
    lds_dma4(psrc == standin ? psrc : psrc + (128 * s + GB * c) / G, &S.prm[wave][0][0]);
    lds_dma4(ssrc == standin ? ssrc : ssrc + static_cast<int64_t>(NSUB) * s, &S.sum[0][0]);
  };
  // the entries and weights of this lane's output tokens 4 c + i
  int64_t eo[4];
  float wo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int sl = 4 * c + i;
    eo[i] = -1;
    wo[i] = 0.0f;
    if (sl < n && k < r) {
      const int p = first + sl;
      eo[i] = ent ? ent[p] : p;
      wo[i] = wgt[p];
    }
  }

  // wave-uniform shape of the wave's rows: planes of the widest packed row,
  // and whether any row is wider than the ring or stored as fp16
  int bw = 0;
#pragma unroll
  for (int t = 0; t < BITSMOE_MAX_BITS; ++t)
    if (__builtin_amdgcn_ballot_w64(packed && ba > t) != 0) bw = t + 1;
  const bool any_raw = __builtin_amdgcn_ballot_w64(ba == 16) != 0;
  // the group's affine step: s and m from the parameter word (packed rows),
  // s = 1, m = 0 for fp16 rows, 0 for rows that contribute nothing
  const float sc_raw = ba == 16 ? 1.0f : 0.0f;

  float z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  // BW: planes decoded, a compile-time bound on the wave's widest packed row;
  // RAW: the wave has fp16 rows
  auto sum_stage = [&]<int BW, bool RAW>(int s, const Stage& S) {
    // the row's plane words of the stage: for sub-group sg, the 32-bit word
    // holding its chunk c (word (sg GB + c CH) / 32 of the stage's four),
    // read at a per-lane LDS address; words of planes the row lacks (or of
    // rows that are not packed) are zeroed here
    uint32_t wd[BITSMOE_MAX_BITS][NSUB];
#pragma unroll
    for (int t = 0; t < BITSMOE_MAX_BITS; ++t)
#pragma unroll
      for (int sg = 0; sg < NSUB; ++sg) wd[t][sg] = 0u;
#pragma unroll
    for (int t = 0; t < RP; ++t) {
      if (t < BW) {
        const uint32_t* row = reinterpret_cast<const uint32_t*>(&S.w[wave][t][rho]);
        const bool has = packed && t < ba;
#pragma unroll
        for (int sg = 0; sg < NSUB; ++sg) {
          const uint32_t v = row[(sg * GB + c * CH) >> 5];
          wd[t][sg] = has ? v : 0u;
        }
      }
    }
    if (BW > RP) {
      // rows of 5..8 bits: the planes past the ring, waited for here
#pragma unroll
      for (int t = RP; t < BITSMOE_MAX_BITS; ++t)
        if (t < BW && packed && t < ba)
#pragma unroll
          for (int sg = 0; sg < NSUB; ++sg)
            wd[t][sg] = pw[2 * t * nw + 4 * s + ((sg * GB + c * CH) >> 5)];
      wait_vmcnt0();
    }
    uint4 raw[4];
    if (RAW) {
      // fp16 rows: the values (the row starts at a 64-bit word: 8-byte loads)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        raw[q] = make_uint4(0, 0, 0, 0);
        if (ba == 16) {
          const int sg = q / SG, qq = q % SG;
          const uint2* p2 = reinterpret_cast<const uint2*>(pw) +
                            ((128 * static_cast<int64_t>(s) + sg * GB + c * CH + 8 * qq) >> 2);
          const uint2 v0 = p2[0], v1 = p2[1];
          raw[q] = make_uint4(v0.x, v0.y, v1.x, v1.y);
        }
      }
      wait_vmcnt0();
    }
#pragma unroll
    for (int sg = 0; sg < NSUB; ++sg) {
      float4v acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int qq = 0; qq < SG; ++qq) {
        const int q = sg * SG + qq;
        // chunk c of step q: bits ((c CH + 8 qq) mod 32) .. +7 of its word
        const int sh = (c * CH + 8 * qq) & 31;
        uint32_t w[BITSMOE_MAX_BITS];
#pragma unroll
        for (int t = 0; t < BITSMOE_MAX_BITS; ++t) w[t] = wd[t][sg];
        half8 a = codes8(w, sh, BW);
        if (RAW && ba == 16) a = __builtin_bit_cast(half8, raw[q]);
        // token rows past TS repeat rows below TS (their sums go unused)
        const int slot = (q * 4 + c) * TS + (rho % TS);
        const half8 h = __builtin_bit_cast(half8, S.x[0][slot]);
        const half8 lo = __builtin_bit_cast(half8, S.x[1][slot]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(h, a, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(lo, a, acc, 0, 0, 0);
      }
      const uint32_t prm = S.prm[wave][sg][rho];
      const float sc = packed ? f16_bits_to_f32(static_cast<uint16_t>(prm & 0xffffu)) : sc_raw;
      const float mn = packed ? f16_bits_to_f32(static_cast<uint16_t>(prm >> 16)) : 0.0f;
      const float4 s4 = S.sum[sg][c];
      const float sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) z[i] = fmaf(sc, acc[i], fmaf(mn, sv[i], z[i]));
    }
  };

#pragma unroll
  for (int j = 0; j < NS - 1; ++j) issue(j, j);
  for (int s0 = 0; s0 < nst; s0 += NS) {
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int s = s0 + j;
      if (s < nst) {
        wait_vmcnt_n<(NS - 2) * PER>();  // this wave's loads of stage s are in
        __syncthreads();                  // everyone's are; stage s - 1 is read
        issue(s + NS - 1, (j + NS - 1) % NS);
        if (any_raw || bw > RP) {
          sum_stage.template operator()<BITSMOE_MAX_BITS, true>(s, st[j]);
        } else {
          switch (bw) {
            case 0:
            case 1: sum_stage.template operator()<1, false>(s, st[j]); break;
            case 2: sum_stage.template operator()<2, false>(s, st[j]); break;
            case 3: sum_stage.template operator()<3, false>(s, st[j]); break;
            default: sum_stage.template operator()<4, false>(s, st[j]); break;
          }
        }
      }
    }
  }
  wait_vmcnt0();  // no load may land in LDS after the workgroup ends
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (eo[i] >= 0) zp[eo[i] * r + k] = wo[i] * z[i];
}

// Z[b][k] for b < Bp, k < rp (zero past B and r) = the sum, in slot order,
// of the token's partial rows zp[slot][k]: slots b kmax + j (pidx null) or
// pidx[b kmax + j] (-1: none).
__global__ __launch_bounds__(256) void zsum_kernel(const float* __restrict__ zp,
                                                   const int64_t* __restrict__ pidx, int kmax,
                                                   int r, int rp, int64_t B, int64_t Bp,
                                                   float* __restrict__ Z) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= Bp * rp) return;
  const int64_t b = idx / rp;
  const int k = static_cast<int>(idx - b * rp);
  float s = 0.0f;
  if (b < B && k < r) {
    for (int j = 0; j < kmax; ++j) {
      const int64_t i = pidx ? pidx[b * kmax + j] : b * kmax + j;
      if (i >= 0) s += zp[i * r + k];
    }
  }
  Z[idx] = s;
}

// Y[b][o] = sum_k Z[b][k] U^T[k][o] for the 64 tokens of blockIdx.y and the
// 16 columns of blockIdx.x as v_mfma_f32_16x16x4_f32 (A = Z, tokens as M;
// B = U^T, columns as N), the 16 waves splitting k into ranges of kw (a
// multiple of 16; Z [Bp][rp] is zero past r) and their sums added in wave
// order through LDS.  Within 16 k's, lane l supplies k = 4 (l / 16) + i at
// sub-step i, so that its four Z values are one float4.
constexpr int kYmmaWaves = 16;
__global__ __launch_bounds__(64 * kYmmaWaves) void decode_ymma_kernel(
    const float* __restrict__ Z, int rp, int r, int kw, const float* __restrict__ Ut,
    int64_t d_out, int64_t B, float* __restrict__ Y) {
  __shared__ float red[kYmmaWaves][16][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tau = lane & 15, c = lane >> 4;
  const int64_t o = static_cast<int64_t>(blockIdx.x) * 16 + tau;
  const int64_t b0 = static_cast<int64_t>(blockIdx.y) * 64;
  const int k0 = wave * kw, k1 = min(k0 + kw, rp);
  float4v acc[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) acc[m] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
  // 64 k's at a time: every load of the four 16-k chunks before their MFMAs
  for (int kb0 = k0; kb0 < k1; kb0 += 64) {
    float4 a[4][4];
    float bv[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int kb = kb0 + 16 * u;
#pragma unroll
      for (int m = 0; m < 4; ++m)
        a[u][m] = kb < k1 ? *reinterpret_cast<const float4*>(Z + (b0 + 16 * m + tau) * rp + kb + 4 * c)
                          : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kk = kb + 4 * c + i;
        bv[u][i] = (kb < k1 && kk < r && o < d_out) ? Ut[static_cast<int64_t>(kk) * d_out + o] : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const float4 am = a[u][m];
          const float av = i == 0 ? am.x : i == 1 ? am.y : i == 2 ? am.z : am.w;
          acc[m] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv[u][i], acc[m], 0, 0, 0);
        }
  }
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][4 * m + i][lane] = acc[m][i];
  __syncthreads();
  const int j = threadIdx.x >> 6, ln = threadIdx.x & 63;
  float sum = 0.0f;
#pragma unroll
  for (int w = 0; w < kYmmaWaves; ++w) sum += red[w][j][ln];
  const int64_t b = b0 + 16 * (j >> 2) + 4 * (ln >> 4) + (j & 3);
  const int64_t col = static_cast<int64_t>(blockIdx.x) * 16 + (ln & 15);
  if (b < B && col < d_out) Y[b * d_out + col] = sum;
}

// ---- input-space form (gate/up): y = sum_j g_j C^_e^T z, z = Phi_r^T x ----

// z[b][k] = sum_i Vt[k][i] X[b][i]: one wave per (k, b).
__global__ __launch_bounds__(256) void zin_kernel(const float* __restrict__ Vt, int r, int64_t d_in,
                                                  const float* __restrict__ X, int64_t B,
                                                  float* __restrict__ z) {
  const int lane = threadIdx.x & 63;
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int64_t b = blockIdx.y;
  if (k >= r || b >= B) return;  // whole wave
  const float* v = Vt + k * d_in;
  const float* x = X + b * d_in;
  float acc = 0.0f;
#pragma unroll 4
  for (int64_t i = lane; i < d_in; i += 64) acc = fmaf(v[i], x[i], acc);
  acc = wave_sum(acc);
  if (lane == 0) z[b * r + k] = acc;
}

// Partial outputs of the routing entries of one job (blockIdx.y; jobs[2j] =
// {expert, first entry, entries 1..T, 0}, jobs[2j+1] = their tokens) over the
// unit rows of row split blockIdx.z:
//   yp[rz][i][o] = w_i sum_{k in split} z[tok_i][k] c^_{e,k}[o].
// Thread (slice rs, segment sg) owns the 32 outputs 32 sg .. 32 sg + 31 of
// segment block blockIdx.x and the rows k = rs, rs + RSL, ... of the split;
// a unit row's 32 entries there are one word of each of its bit planes and
// one group parameter, so c^ = q s + m is summed as (z s) q and z m.  The
// RSL slices are added in slice order through LDS.
template <int T>
__global__ __launch_bounds__(256) void yin_kernel(
    const uint32_t* __restrict__ codes32, const uint32_t* __restrict__ params,
    const uint8_t* __restrict__ bits, const int64_t* __restrict__ off, int64_t total_words,
    int r, int d, int G, int SEGW, int rows_split, const float* __restrict__ z,
    const int4* __restrict__ jobs, const float* __restrict__ ew, int64_t nnz,
    float* __restrict__ yp) {
  __shared__ float red[256 * kSeg];
  const int4 job = jobs[2 * blockIdx.y];
  const int4 jt = jobs[2 * blockIdx.y + 1];
  const int e = job.x;
  const int64_t i0 = job.y;
  const int nt = job.z;
  const int tk[4] = {jt.x, jt.y, jt.z, jt.w};
  const int RSL = 256 / SEGW;
  const int sg_local = threadIdx.x % SEGW, rs = threadIdx.x / SEGW;
  const int nseg = d / kSeg;
  const int sg = static_cast<int>(blockIdx.x) * SEGW + sg_local;
  const int64_t nw = d / 64;
  const int kb = static_cast<int>(blockIdx.z) * rows_split;
  const int ke = min(r, kb + rows_split);
  float acc[T][kSeg], macc[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    macc[t] = 0.0f;
#pragma unroll
    for (int j = 0; j < kSeg; ++j) acc[t][j] = 0.0f;
  }
  if (sg < nseg) {
    for (int k = kb + rs; k < ke; k += RSL) {
      const int64_t u = static_cast<int64_t>(e) * r + k;
      const int b = bits[u];
      const int64_t o0 = off[u], o1 = off[u + 1];
      // a unit whose width or offsets are inconsistent contributes nothing
      if (!(width_ok(b) && b != 0 && o1 - o0 == b * nw && o0 >= 0 && o1 <= total_words)) continue;
      float zk[T];
#pragma unroll
      for (int t = 0; t < T; ++t) zk[t] = t < nt ? z[static_cast<int64_t>(tk[t]) * r + k] : 0.0f;
      if (b == 16) {
        const uint2* h = reinterpret_cast<const uint2*>(codes32 + 2 * o0) + 8 * sg;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const uint2 v = h[q];
          const float c[4] = {f16_bits_to_f32(static_cast<uint16_t>(v.x & 0xffffu)),
                              f16_bits_to_f32(static_cast<uint16_t>(v.x >> 16)),
                              f16_bits_to_f32(static_cast<uint16_t>(v.y & 0xffffu)),
                              f16_bits_to_f32(static_cast<uint16_t>(v.y >> 16))};
#pragma unroll
          for (int c4 = 0; c4 < 4; ++c4)
#pragma unroll
            for (int t = 0; t < T; ++t) acc[t][4 * q + c4] = fmaf(zk[t], c[c4], acc[t][4 * q + c4]);
        }
        continue;
      }
      const uint32_t prm = params[u * (d / G) + (sg * kSeg) / G];
      const float s = f16_bits_to_f32(static_cast<uint16_t>(prm & 0xffffu));
      const float m = f16_bits_to_f32(static_cast<uint16_t>(prm >> 16));
      const uint32_t* pw = codes32 + 2 * o0 + sg;  // plane t: word 2 (o0 + t nw) + sg
      uint32_t qb[kSeg / 4];
      {
        const uint32_t p0 = pw[0];
#pragma unroll
        for (int kk = 0; kk < kSeg / 4; ++kk) qb[kk] = spread4(p0 >> (4 * kk));
      }
      for (int t = 1; t < b; ++t) {
        const uint32_t pt = pw[2 * t * nw];
#pragma unroll
        for (int kk = 0; kk < kSeg / 4; ++kk) qb[kk] |= spread4(pt >> (4 * kk)) << t;
      }
      float zs[T];
#pragma unroll
      for (int t = 0; t < T; ++t) {
        zs[t] = zk[t] * s;
        macc[t] = fmaf(zk[t], m, macc[t]);
      }
#pragma unroll
      for (int kk = 0; kk < kSeg / 4; ++kk)
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const float q = static_cast<float>((qb[kk] >> (8 * c4)) & 0xffu);
#pragma unroll
          for (int t = 0; t < T; ++t) acc[t][4 * kk + c4] = fmaf(zs[t], q, acc[t][4 * kk + c4]);
        }
    }
  }
  // slices in order, one token at a time: red[rs][sg_local][j]
#pragma unroll
  for (int t = 0; t < T; ++t) {
    if (t >= nt) continue;  // uniform over the workgroup
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kSeg; ++j) red[(rs * SEGW + sg_local) * kSeg + j] = acc[t][j] + macc[t];
    __syncthreads();
    const float wt = ew[i0 + t];
    for (int idx = threadIdx.x; idx < SEGW * kSeg; idx += 256) {
      const int sgl = idx / kSeg, j = idx - sgl * kSeg;
      const int sgo = static_cast<int>(blockIdx.x) * SEGW + sgl;
      if (sgo >= nseg) continue;
      float v = 0.0f;
      for (int q = 0; q < RSL; ++q) v += red[(q * SEGW + sgl) * kSeg + j];
      yp[(static_cast<int64_t>(blockIdx.z) * nnz + i0 + t) * d + static_cast<int64_t>(sgo) * kSeg + j] =
          wt * v;
    }
  }
}

// y[b][o] = the sum of the partials yp[rz][i][o] over the row splits rz and
// token b's routing entries i: P = nsplit kmax partials per output.  A
// workgroup covers 64 outputs of one token; token b's entry list is staged
// in LDS first, then its four waves take the partials p = w mod 4 with 16
// accumulators each (16 independent loads in flight), combined in a fixed
// order through LDS.
__global__ __launch_bounds__(256) void ysum_kernel(const float* __restrict__ yp, int nsplit,
                                                   int64_t nnz, const int64_t* __restrict__ pidx,
                                                   int kmax, int64_t d, int64_t B,
                                                   float* __restrict__ Y) {
  constexpr int U = 16;
  __shared__ float red[4][64];
  __shared__ int64_t ent[1024];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t o = static_cast<int64_t>(blockIdx.x) * 64 + lane;
  const int64_t b = blockIdx.y;
  float a[U];
#pragma unroll
  for (int q = 0; q < U; ++q) a[q] = 0.0f;
  for (int j0 = 0; j0 < kmax; j0 += 1024) {  // entry lists longer than 1024: in pieces
    const int nj = min(1024, kmax - j0);
    __syncthreads();
    for (int j = threadIdx.x; j < nj; j += 256) ent[j] = pidx[b * kmax + j0 + j];
    __syncthreads();
    const int P = nsplit * nj;
    if (o < d) {
      for (int p0 = wave; p0 < P; p0 += 4 * U) {
#pragma unroll
        for (int q = 0; q < U; ++q) {
          const int p = p0 + 4 * q;
          if (p < P) {
            const int j = p / nsplit, sp = p - j * nsplit;
            const int64_t i = ent[j];
            if (i >= 0) a[q] += yp[(sp * nnz + i) * d + o];
          }
        }
      }
    }
  }
  float t = 0.0f;
#pragma unroll
  for (int q = 0; q < U; ++q) t += a[q];
  red[wave][lane] = t;
  __syncthreads();
  if (wave == 0 && o < d) Y[b * d + o] = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
}

}  // namespace
}  // namespace bitsmoe

namespace bitsmoe {
namespace {

bitsmoe_status check_decode(const char* who, const void* codes, const void* params,
                            const void* bits, const void* offs, const void* Ut, const void* X,
                            const void* Y, int64_t total_words, int64_t E, int64_t r, int64_t d_in,
                            int group, int64_t d_out, int64_t B) {
  // the message text is only built on failure (no host allocation on success)
  auto bad = [who](bitsmoe_status st, const char* msg) { return fail(st, std::string(who) + msg); };
  if (!codes || !params || !bits || !offs || !Ut || !X || !Y)
    return bad(BITSMOE_ERR_ARG, ": null pointer");
  if (!aligned16({codes, params, bits, offs, Ut, X, Y}))
    return bad(BITSMOE_ERR_ARG, ": device pointers must be 16-byte aligned");
  if (E <= 0 || r <= 0 || d_in <= 0 || d_out <= 0 || B <= 0 || total_words < 0)
    return bad(BITSMOE_ERR_ARG, ": non-positive size");
  if (E > 65535 || B > 65535) return bad(BITSMOE_ERR_SHAPE, ": at most 65535 experts and tokens");
  if (!(group == 32 || group == 64 || group == 128 || group == 256))
    return bad(BITSMOE_ERR_SHAPE, ": group must be 32, 64, 128 or 256");
  if (d_in % 64 != 0 || d_in % group != 0)
    return bad(BITSMOE_ERR_SHAPE, ": the units' length must be a multiple of 64 and of the group");
  if (r > 8192) return bad(BITSMOE_ERR_SHAPE, ": r above 8192");
  if (d_in > (1 << 20)) return bad(BITSMOE_ERR_SHAPE, ": the units' length is above 2^20");
  return ok();
}

// Host routing grouped by expert, checked, with each token's entries (in the
// order given) and the experts' entries in jobs of up to T (tmax when some
// expert has several tokens, else 1).
struct RoutingTables {
  int64_t nnz = 0, kmax = 1, njobs = 0;
  int T = 1;
  std::vector<int64_t> pidx;   // [B][kmax], -1 = none
  std::vector<int32_t> jobs;   // per job: {expert, first entry, entries, 0}, {tokens}
};

bitsmoe_status build_routing(const std::string& who, int64_t E, int64_t B,
                             const int64_t* offsets_host, const int32_t* tokens_host,
                             const float* weights_host, int tmax, RoutingTables* rt) {
  if (!offsets_host || !tokens_host || !weights_host) return fail(BITSMOE_ERR_ARG, who + ": null pointer");
  if (offsets_host[0] != 0) return fail(BITSMOE_ERR_ARG, who + ": offsets[0] must be 0");
  for (int64_t e = 0; e < E; ++e)
    if (offsets_host[e + 1] < offsets_host[e])
      return fail(BITSMOE_ERR_ARG, who + ": offsets must not decrease");
  const int64_t nnz = offsets_host[E];
  if (nnz > INT32_MAX) return fail(BITSMOE_ERR_SHAPE, who + ": too many routing entries");
  std::vector<int64_t> cnt(static_cast<size_t>(B), 0);
  for (int64_t i = 0; i < nnz; ++i) {
    if (tokens_host[i] < 0 || tokens_host[i] >= B)
      return fail(BITSMOE_ERR_ARG, who + ": token index outside [0, B)");
    if (!std::isfinite(weights_host[i])) return fail(BITSMOE_ERR_ARG, who + ": non-finite weight");
    ++cnt[static_cast<size_t>(tokens_host[i])];
  }
  int64_t kmax = 1;
  for (int64_t c : cnt) kmax = std::max(kmax, c);
  if (kmax > 65535) return fail(BITSMOE_ERR_SHAPE, who + ": more than 65535 entries of one token");
  rt->pidx.assign(static_cast<size_t>(B * kmax), -1);
  std::fill(cnt.begin(), cnt.end(), 0);
  for (int64_t i = 0; i < nnz; ++i) {
    const int64_t b = tokens_host[i];
    rt->pidx[static_cast<size_t>(b * kmax + cnt[static_cast<size_t>(b)]++)] = i;
  }
  int64_t cmax = 0;
  for (int64_t e = 0; e < E; ++e) cmax = std::max(cmax, offsets_host[e + 1] - offsets_host[e]);
  const int T = cmax > 1 ? tmax : 1;
  rt->jobs.clear();
  for (int64_t e = 0; e < E; ++e)
    for (int64_t i = offsets_host[e]; i < offsets_host[e + 1]; i += T) {
      const int64_t n = std::min<int64_t>(T, offsets_host[e + 1] - i);
      rt->jobs.push_back(static_cast<int32_t>(e));
      rt->jobs.push_back(static_cast<int32_t>(i));
      rt->jobs.push_back(static_cast<int32_t>(n));
      rt->jobs.push_back(0);
      for (int t = 0; t < 4; ++t) rt->jobs.push_back(t < n ? tokens_host[i + t] : 0);
    }
  rt->njobs = static_cast<int64_t>(rt->jobs.size() / 8);
  if (rt->njobs > 65535) return fail(BITSMOE_ERR_SHAPE, who + ": more than 65535 routing chunks");
  rt->nnz = nnz;
  rt->kmax = kmax;
  rt->T = T;
  return ok();
}

// Device copies of the jobs [njobs][8], the weights [nnz] and the token entry
// lists [B][kmax] in the small-table scratch; waits for the stream (the host
// tables may go away after the call returns).
bitsmoe_status upload_routing(const std::string& who, const RoutingTables& rt,
                              const float* weights_host, int64_t B, void* stream, int4** jobs_d,
                              int64_t** pidx_d, float** w_d) {
  bitsmoe_status st;
  const size_t job_bytes = static_cast<size_t>(std::max<int64_t>(rt.njobs, 1)) * 32;
  const size_t pidx_bytes = static_cast<size_t>(B * rt.kmax) * 8;
  const size_t w_bytes = (static_cast<size_t>(rt.nnz) * 4 + 15) / 16 * 16;
  char* tab = static_cast<char*>(scratch(kScratchMisc, job_bytes + pidx_bytes + w_bytes + 64, stream, &st));
  if (!tab) return st;
  *jobs_d = reinterpret_cast<int4*>(tab);
  *pidx_d = reinterpret_cast<int64_t*>(tab + job_bytes);
  *w_d = reinterpret_cast<float*>(tab + job_bytes + pidx_bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t he = hipSuccess;
  if (rt.njobs > 0) he = hipMemcpyAsync(*jobs_d, rt.jobs.data(), rt.njobs * 32, hipMemcpyHostToDevice, s);
  if (he == hipSuccess)
    he = hipMemcpyAsync(*pidx_d, rt.pidx.data(), B * rt.kmax * 8, hipMemcpyHostToDevice, s);
  if (he == hipSuccess && rt.nnz > 0)
    he = hipMemcpyAsync(*w_d, weights_host, rt.nnz * 4, hipMemcpyHostToDevice, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) return device_error((who + ": routing table copy").c_str(), he);
  return ok();
}

// Launch shape of both kernels.
struct DecodeGeom {
  int L;            // lanes per unit row (power of two, <= 64)
  bool one_slice;   // the row's segments fit in L lanes
  int R;            // rows per wave pass
  int passes;       // passes per wave
  int64_t rows_wg;  // rows per decode_z workgroup
  int64_t rp;       // r padded for decode_y
  int TB;           // tokens per decode_y workgroup
};

DecodeGeom decode_geometry(int64_t njobs, int64_t r, int64_t d_in, int64_t B) {
  DecodeGeom g;
  // lanes per row: the row's segments rounded up to a power of two (up to 64)
  const int nseg = static_cast<int>(d_in / 32);
  g.L = 2;
  while (g.L < nseg && g.L < 64) g.L *= 2;
  g.one_slice = nseg <= g.L;
  g.R = 64 / g.L;
  // rows per wave: about 1024 waves or more, up to 8 (and L) passes of R
  // rows; more passes reuse the token values held in registers
  const int64_t total_rows = std::max<int64_t>(njobs, 1) * r;
  g.passes = static_cast<int>(
      std::clamp<int64_t>(total_rows / (g.R * 1024), 1, std::min(8, g.one_slice ? g.L : 8)));
  g.rows_wg = static_cast<int64_t>(kWaves) * g.passes * g.R;
  // decode_y: token tile TB with z [TB][rp] and the partials within 64 KiB
  // of LDS (rp = r rounded up to 16 waves x a multiple of 4 rows)
  g.rp = ((r + kYWaves - 1) / kYWaves + 3) / 4 * 4 * kYWaves;
  g.TB = 8;
  while (g.TB > 1 && static_cast<int64_t>(g.TB) * (g.rp + kYWaves * 64) * 4 > 65536) g.TB /= 2;
  if (B == 1) g.TB = 1;
  return g;
}

bitsmoe_status decode_launch(const DecodeGeom& g, int T, bool topk_jobs, int64_t njobs,
                             const uint64_t* codes_dev, const uint16_t* params_dev,
                             const uint8_t* bits_dev, const int64_t* offs_dev, int64_t total_words,
                             int64_t E, int64_t r, int64_t d_in, int group, const float* Ut_dev,
                             int64_t d_out, const float* X_dev, int64_t B, const int4* jobs_d,
                             const int32_t* topk_d, int kk, const float* w_d, const int64_t* pidx_d,
                             int kmax, float* zp, float* Y_dev, hipStream_t s,
                             bool timed = true) {
  const uint32_t* pr = reinterpret_cast<const uint32_t*>(params_dev);
  const uint32_t* c32 = reinterpret_cast<const uint32_t*>(codes_dev);
  // without timing the launches create no events
  void* stream = s;
  const char* zname = timed ? "moe_decode_z" : nullptr;
  const char* yname = timed ? "moe_decode_y" : nullptr;
  if (njobs > 0) {
    KernelTimer timer(zname, stream);
    dim3 grid(static_cast<unsigned>((r + g.rows_wg - 1) / g.rows_wg), static_cast<unsigned>(njobs));
#define BITSMOE_DEC(TT, OS, TK)                                                                    \
  hipLaunchKernelGGL((decode_z_kernel<TT, OS, TK>), grid, dim3(64 * kWaves), 0, s, c32, pr,        \
                     bits_dev, offs_dev, total_words, static_cast<int>(r), static_cast<int>(d_in), \
                     group, g.L, g.passes, X_dev, jobs_d, topk_d, kk, static_cast<int>(E), w_d, zp)
    if (topk_jobs) {
      if (g.one_slice) BITSMOE_DEC(1, true, true); else BITSMOE_DEC(1, false, true);
    } else if (T == 2) {
      if (g.one_slice) BITSMOE_DEC(2, true, false); else BITSMOE_DEC(2, false, false);
    } else {
      if (g.one_slice) BITSMOE_DEC(1, true, false); else BITSMOE_DEC(1, false, false);
    }
#undef BITSMOE_DEC
  }
  BITSMOE_LAUNCH_CHECK("moe_decode: z launch");
  {
    KernelTimer timer(yname, stream);
    dim3 grid(static_cast<unsigned>((d_out + 63) / 64), static_cast<unsigned>((B + g.TB - 1) / g.TB));
    const size_t lds = static_cast<size_t>(g.TB) * (g.rp + kYWaves * 64) * 4;
#define BITSMOE_DECY(TT)                                                                   \
  hipLaunchKernelGGL(decode_y_kernel<TT>, grid, dim3(64 * kYWaves), lds, s, zp, pidx_d,    \
                     kmax, static_cast<int>(r), Ut_dev, d_out, B, Y_dev)
    switch (g.TB) {
      case 8: BITSMOE_DECY(8); break;
      case 4: BITSMOE_DECY(4); break;
      case 2: BITSMOE_DECY(2); break;
      default: BITSMOE_DECY(1); break;
    }
#undef BITSMOE_DECY
  }
  BITSMOE_LAUNCH_CHECK("moe_decode: y launch");
  return ok();
}

// Batches from this many tokens take the matrix-core z step (at one token
// the VALU form, which waits on fewer dependent loads, is faster), when the
// units' length is a multiple of its 128-entry stages.
constexpr int64_t kMmaMinTokens = 16;
bool mma_path(int64_t B, int64_t d_in) { return B >= kMmaMinTokens && d_in % 128 == 0; }

// Tokens per job of the z step: 8 while the experts average at most 8
// routing entries (the ring's x stage is then half the size, which leaves
// room for three workgroups per CU), else 16.
int mma_job_tokens(int64_t E, int64_t nnz) {
  const int64_t busy = std::max<int64_t>(std::min(E, nnz), 1);
  return nnz <= 8 * busy ? 8 : 16;
}

// Bytes of scratch decode_mma needs: x as fp16 hi/lo, the block sums, the
// job table and its count, the sorted entries, tokens and weights, the
// partials and the token sums Z [Bp][rp] (each region 256-byte aligned).
struct MmaScratch {
  size_t xb, sb, jb, eb, zb, Zb;
  int64_t max_jobs, Bp, rp;
  size_t total() const { return 2 * xb + sb + jb + 3 * eb + zb + Zb; }
};
MmaScratch mma_scratch(int64_t E, int64_t r, int64_t d_in, int group, int64_t B, bool topk,
                       int64_t nnz, int64_t njobs_host) {
  auto up = [](size_t b) { return (b + 255) / 256 * 256; };
  MmaScratch m;
  // jobs: one per expert with routing entries, plus one per further jt
  const int jt = mma_job_tokens(E, nnz);
  m.max_jobs = topk ? std::min<int64_t>(E, nnz) + (nnz + jt - 1) / jt : njobs_host;
  m.Bp = (B + 63) / 64 * 64;
  m.rp = (r + 15) / 16 * 16;
  m.xb = up(static_cast<size_t>(B * d_in) * 2);
  m.sb = up(static_cast<size_t>(B * (d_in / std::min(group, 128))) * 4);
  m.jb = up(static_cast<size_t>(std::max<int64_t>(m.max_jobs, 1)) * 16 + 16);
  m.eb = up(static_cast<size_t>(std::max<int64_t>(nnz, 1)) * 4);
  m.zb = up(static_cast<size_t>(std::max<int64_t>(nnz, 1) * r) * 4);
  m.Zb = up(static_cast<size_t>(m.Bp * m.rp) * 4);
  return m;
}

// The matrix-core z step and the y step for B tokens, routing already in
// device tables (jobs, ent, tok, wgt; njobs on the device when not null) or
// produced from a device top-k table (topk set: prep_kernel).  The
// scratch of mma_scratch is `base` when given (the caller checked its size),
// else the library's scratch cache; `timed` records kernel events.
bitsmoe_status decode_mma(const uint32_t* c32, const uint32_t* pr, const uint8_t* bits_dev,
                          const int64_t* offs_dev, int64_t total_words, int64_t E, int64_t r,
                          int64_t d_in, int group, const float* Ut_dev, int64_t d_out,
                          const float* X_dev, int64_t B, const int32_t* topk, const float* topw,
                          int kk, int64_t nnz, const int4* jobs_in, int64_t njobs_host,
                          const int32_t* tok_in, const float* wgt_in, const int64_t* pidx_d,
                          int kmax, float* Y_dev, void* stream, char* base = nullptr,
                          bool timed = true) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int ng = static_cast<int>(d_in / group);
  const MmaScratch m = mma_scratch(E, r, d_in, group, B, topk != nullptr, nnz, njobs_host);
  const int64_t max_jobs = m.max_jobs;
  const size_t xb = m.xb, sb = m.sb, jb = m.jb, eb = m.eb;
  bitsmoe_status st;
  char* sp = base;
  if (!sp) {
    sp = static_cast<char*>(scratch(kScratchPart, m.total(), stream, &st));
    if (!sp) return st;
  }
  _Float16* xh = reinterpret_cast<_Float16*>(sp);
  _Float16* xl = reinterpret_cast<_Float16*>(sp + xb);
  float* xs = reinterpret_cast<float*>(sp + 2 * xb);
  int4* jobs = reinterpret_cast<int4*>(sp + 2 * xb + sb);
  int* njobs = reinterpret_cast<int*>(sp + 2 * xb + sb + jb - 16);
  int32_t* ent = reinterpret_cast<int32_t*>(sp + 2 * xb + sb + jb);
  int32_t* tok = reinterpret_cast<int32_t*>(sp + 2 * xb + sb + jb + eb);
  float* wgt = reinterpret_cast<float*>(sp + 2 * xb + sb + jb + 2 * eb);
  float* zp = reinterpret_cast<float*>(sp + 2 * xb + sb + jb + 3 * eb);
  float* Zs = reinterpret_cast<float*>(sp + 2 * xb + sb + jb + 3 * eb + m.zb);
  const int gb = std::min(group, 128);
  const int jt = mma_job_tokens(E, nnz);
  {
    // one launch: routing (top-k form) in workgroup 0, x prep in the others
    KernelTimer timer(timed ? "moe_decode_prep" : nullptr, stream);
    const int64_t nblk = B * (d_in / gb);
    const unsigned nwg = static_cast<unsigned>((nblk + 15) / 16) + (topk ? 1u : 0u);
    hipLaunchKernelGGL(prep_kernel, dim3(nwg), dim3(kRouteThreads), 0, s, topk, topw, nnz, kk,
                       static_cast<int>(E), static_cast<int>(r), jt, jobs, njobs, ent, tok, wgt, zp,
                       X_dev, nblk, static_cast<int>(d_in), gb, xh, xl, xs);
  }
  BITSMOE_LAUNCH_CHECK("moe_decode: prep launch");
  if (max_jobs > 0) {
    KernelTimer timer(timed ? "moe_decode_z" : nullptr, stream);
    constexpr int kRows = 16 * kMmaWaves;
    dim3 grid(static_cast<unsigned>((r + kRows - 1) / kRows), static_cast<unsigned>(max_jobs));
#define BITSMOE_DECZ(GG, TT)                                                                     \
  hipLaunchKernelGGL((decode_zmma_kernel<GG, TT, kMmaWaves, kMmaStages>), grid, dim3(64 * kMmaWaves), \
                     0, s, c32, pr, bits_dev, offs_dev, total_words, static_cast<int>(r),         \
                     static_cast<int>(d_in), xh, xl, xs, topk ? jobs : jobs_in,                   \
                     topk ? njobs : nullptr, topk ? ent : nullptr, topk ? tok : tok_in,           \
                     topk ? wgt : wgt_in, zp)
#define BITSMOE_DECZ_G(GG) \
  if (jt == 8) BITSMOE_DECZ(GG, 8); else BITSMOE_DECZ(GG, 16);
    switch (group) {
      case 32: BITSMOE_DECZ_G(32); break;
      case 64: BITSMOE_DECZ_G(64); break;
      case 128: BITSMOE_DECZ_G(128); break;
      default: BITSMOE_DECZ_G(256); break;
    }
#undef BITSMOE_DECZ_G
#undef BITSMOE_DECZ
  }
  BITSMOE_LAUNCH_CHECK("moe_decode: z launch");
  {
    // the y step: token sums (zsum), then y = U z (decode_ymma)
    KernelTimer timer(timed ? "moe_decode_y" : nullptr, stream);
    const int64_t nz = m.Bp * m.rp;
    hipLaunchKernelGGL(zsum_kernel, dim3(static_cast<unsigned>((nz + 255) / 256)), dim3(256), 0, s,
                       zp, pidx_d, kmax, static_cast<int>(r), static_cast<int>(m.rp), B, m.Bp, Zs);
    const int kw = static_cast<int>((m.rp / 16 + kYmmaWaves - 1) / kYmmaWaves * 16);
    dim3 grid(static_cast<unsigned>((d_out + 15) / 16), static_cast<unsigned>(m.Bp / 64));
    hipLaunchKernelGGL(decode_ymma_kernel, grid, dim3(64 * kYmmaWaves), 0, s, Zs,
                       static_cast<int>(m.rp), static_cast<int>(r), kw, Ut_dev, d_out, B, Y_dev);
  }
  BITSMOE_LAUNCH_CHECK("moe_decode: y launch");
  return ok();
}

// The top-k decode without allocation keeps its scratch (the partial sums;
// on the matrix-core path also x as fp16, the group sums and the routing
// tables) in a fixed device array, decode_partials below: every GPU the
// library runs on holds one copy (16 MiB) until the process ends.  Its address differs per device
// and is looked up once per device, with that device current; host code
// uses only that address (the array's name is a host-side stand-in).
constexpr int64_t kNoAllocPartials = int64_t{1} << 22;  // floats (16 MiB)
constexpr int kNoAllocMaxDevices = 64;

}  // namespace
}  // namespace bitsmoe

static __device__ __align__(256) float decode_partials[bitsmoe::kNoAllocPartials];

namespace bitsmoe {
namespace {

std::mutex g_partials_mu;
float* g_partials[kNoAllocMaxDevices];  // device address of decode_partials, per device

// The current device's copy of decode_partials (looked up on the first call
// on that device).  Allocates nothing.
bitsmoe_status device_partials(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return device_error("moe_decode_topk_noalloc: hipGetDevice", e);
  if (dev < 0 || dev >= kNoAllocMaxDevices)
    return fail(BITSMOE_ERR_DEVICE, "moe_decode_topk_noalloc: device index above 63");
  std::lock_guard<std::mutex> lock(g_partials_mu);
  if (!g_partials[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(decode_partials));
    if (e != hipSuccess || !p)
      return device_error("moe_decode_topk_noalloc: hipGetSymbolAddress", e != hipSuccess ? e : hipErrorUnknown);
    g_partials[dev] = static_cast<float*>(p);
  }
  *out = g_partials[dev];
  return BITSMOE_OK;
}

// Checks of the top-k table shared by both top-k entry points.
bitsmoe_status check_topk(const char* who, const void* topk_experts, const void* topk_weights,
                          int64_t E, int64_t B, int64_t k) {
  auto bad = [who](bitsmoe_status st, const char* msg) { return fail(st, std::string(who) + msg); };
  if (!topk_experts || !topk_weights) return bad(BITSMOE_ERR_ARG, ": null pointer");
  if (!aligned16({topk_experts, topk_weights}))
    return bad(BITSMOE_ERR_ARG, ": device pointers must be 16-byte aligned");
  if (k <= 0) return bad(BITSMOE_ERR_ARG, ": non-positive k");
  if (k > E || B * k > 65535)
    return bad(BITSMOE_ERR_SHAPE, ": k above E, or more than 65535 routing slots");
  return BITSMOE_OK;
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
  bitsmoe_status st = check_decode("moe_decode", codes_dev, params_dev, bits_dev, word_offsets_dev,
                                   Ut_dev, X_dev, Y_dev, total_words, E, r, d_in, group, d_out, B);
  if (st != BITSMOE_OK) return st;
  RoutingTables rt;
  // two tokens per job: the token values a lane holds take 64 registers
  // (four tokens' 128 left room for two waves per SIMD only)
  st = build_routing("moe_decode", E, B, offsets_host, tokens_host, weights_host, 2, &rt);
  if (st != BITSMOE_OK) return st;
  if (mma_path(B, d_in)) {
    // matrix-core z step: jobs of up to jt consecutive entries of an expert
    // (the entries are grouped by expert, so a position is its entry)
    const int jt = mma_job_tokens(E, rt.nnz);
    std::vector<int4> jobs4;
    for (int64_t e = 0; e < E; ++e)
      for (int64_t i = offsets_host[e]; i < offsets_host[e + 1]; i += jt)
        jobs4.push_back(make_int4(static_cast<int>(e), static_cast<int>(i),
                                  static_cast<int>(std::min<int64_t>(jt, offsets_host[e + 1] - i)), 0));
    const size_t jbytes = (jobs4.size() * 16 + 255) / 256 * 256;
    const size_t ebytes = (static_cast<size_t>(std::max<int64_t>(rt.nnz, 1)) * 4 + 255) / 256 * 256;
    const size_t pbytes = static_cast<size_t>(B * rt.kmax) * 8;
    char* tab = static_cast<char*>(scratch(kScratchMisc, jbytes + 2 * ebytes + pbytes + 256, stream, &st));
    if (!tab) return st;
    int4* jobs_d = reinterpret_cast<int4*>(tab);
    int32_t* tok_d = reinterpret_cast<int32_t*>(tab + jbytes);
    float* w_d = reinterpret_cast<float*>(tab + jbytes + ebytes);
    int64_t* pidx_d = reinterpret_cast<int64_t*>(tab + jbytes + 2 * ebytes);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t he = hipSuccess;
    if (!jobs4.empty()) he = hipMemcpyAsync(jobs_d, jobs4.data(), jobs4.size() * 16, hipMemcpyHostToDevice, s);
    if (he == hipSuccess && rt.nnz > 0)
      he = hipMemcpyAsync(tok_d, tokens_host, rt.nnz * 4, hipMemcpyHostToDevice, s);
    if (he == hipSuccess && rt.nnz > 0)
      he = hipMemcpyAsync(w_d, weights_host, rt.nnz * 4, hipMemcpyHostToDevice, s);
    if (he == hipSuccess) he = hipMemcpyAsync(pidx_d, rt.pidx.data(), pbytes, hipMemcpyHostToDevice, s);
    if (he == hipSuccess) he = hipStreamSynchronize(s);  // the host tables go away on return
    if (he != hipSuccess) return device_error("moe_decode: routing table copy", he);
    return decode_mma(reinterpret_cast<const uint32_t*>(codes_dev),
                      reinterpret_cast<const uint32_t*>(params_dev), bits_dev, word_offsets_dev,
                      total_words, E, r, d_in, group, Ut_dev, d_out, X_dev, B, nullptr, nullptr, 1,
                      rt.nnz, jobs_d, static_cast<int64_t>(jobs4.size()), tok_d, w_d, pidx_d,
                      static_cast<int>(rt.kmax), Y_dev, stream);
  }
  const DecodeGeom g = decode_geometry(rt.njobs, r, d_in, B);
  int4* jobs_d;
  int64_t* pidx_d;
  float* w_d;
  st = upload_routing("moe_decode", rt, weights_host, B, stream, &jobs_d, &pidx_d, &w_d);
  if (st != BITSMOE_OK) return st;
  // partials zp [nnz][r]
  float* zp = static_cast<float*>(scratch(kScratchPart, std::max<int64_t>(rt.nnz, 1) * r * 4, stream, &st));
  if (!zp) return st;
  return decode_launch(g, rt.T, false, rt.njobs, codes_dev, params_dev, bits_dev, word_offsets_dev,
                       total_words, E, r, d_in, group, Ut_dev, d_out, X_dev, B, jobs_d, nullptr, 1,
                       w_d, pidx_d, static_cast<int>(rt.kmax), zp, Y_dev,
                       static_cast<hipStream_t>(stream));
}

extern "C" bitsmoe_status bitsmoe_moe_decode_topk(const uint64_t* codes_dev, const uint16_t* params_dev,
                                                  const uint8_t* bits_dev,
                                                  const int64_t* word_offsets_dev, int64_t total_words,
                                                  int64_t E, int64_t r, int64_t d_in, int group,
                                                  const float* Ut_dev, int64_t d_out,
                                                  const float* X_dev, int64_t B, int64_t k,
                                                  const int32_t* topk_experts_dev,
                                                  const float* topk_weights_dev, float* Y_dev,
                                                  void* stream) {
  bitsmoe_status st = check_decode("moe_decode_topk", codes_dev, params_dev, bits_dev,
                                   word_offsets_dev, Ut_dev, X_dev, Y_dev, total_words, E, r, d_in,
                                   group, d_out, B);
  if (st != BITSMOE_OK) return st;
  st = check_topk("moe_decode_topk", topk_experts_dev, topk_weights_dev, E, B, k);
  if (st != BITSMOE_OK) return st;
  if (mma_path(B, d_in) && E <= kRouteMaxExperts)
    return decode_mma(reinterpret_cast<const uint32_t*>(codes_dev),
                      reinterpret_cast<const uint32_t*>(params_dev), bits_dev, word_offsets_dev,
                      total_words, E, r, d_in, group, Ut_dev, d_out, X_dev, B, topk_experts_dev,
                      topk_weights_dev, static_cast<int>(k), B * k, nullptr, 0, nullptr, nullptr,
                      nullptr, static_cast<int>(k), Y_dev, stream);
  const int64_t njobs = B * k;
  const DecodeGeom g = decode_geometry(njobs, r, d_in, B);
  float* zp = static_cast<float*>(scratch(kScratchPart, njobs * r * 4, stream, &st));
  if (!zp) return st;
  return decode_launch(g, 1, true, njobs, codes_dev, params_dev, bits_dev, word_offsets_dev,
                       total_words, E, r, d_in, group, Ut_dev, d_out, X_dev, B, nullptr,
                       topk_experts_dev, static_cast<int>(k), topk_weights_dev, nullptr,
                       static_cast<int>(k), zp, Y_dev, static_cast<hipStream_t>(stream));
}

extern "C" bitsmoe_status bitsmoe_moe_decode_topk_noalloc(
    const uint64_t* codes_dev, const uint16_t* params_dev, const uint8_t* bits_dev,
    const int64_t* word_offsets_dev, int64_t total_words, int64_t E, int64_t r, int64_t d_in,
    int group, const float* Ut_dev, int64_t d_out, const float* X_dev, int64_t B, int64_t k,
    const int32_t* topk_experts_dev, const float* topk_weights_dev, float* Y_dev, void* stream) {
  bitsmoe_status st = check_decode("moe_decode_topk_noalloc", codes_dev, params_dev, bits_dev,
                                   word_offsets_dev, Ut_dev, X_dev, Y_dev, total_words, E, r, d_in,
                                   group, d_out, B);
  if (st != BITSMOE_OK) return st;
  st = check_topk("moe_decode_topk_noalloc", topk_experts_dev, topk_weights_dev, E, B, k);
  if (st != BITSMOE_OK) return st;
  const int64_t njobs = B * k;
  const bool mma = mma_path(B, d_in) && E <= kRouteMaxExperts;
  // the same path as bitsmoe_moe_decode_topk, with every scratch region in
  // the fixed array
  const size_t need = mma ? mma_scratch(E, r, d_in, group, B, true, njobs, 0).total()
                          : static_cast<size_t>(njobs * r) * sizeof(float);
  if (need > static_cast<size_t>(kNoAllocPartials) * sizeof(float))
    return fail(BITSMOE_ERR_SHAPE,
                "moe_decode_topk_noalloc: the call needs more than the fixed scratch buffer (16 MiB)");
  float* zp = nullptr;
  st = device_partials(&zp);
  if (st != BITSMOE_OK) return st;
  if (mma)
    return decode_mma(reinterpret_cast<const uint32_t*>(codes_dev),
                      reinterpret_cast<const uint32_t*>(params_dev), bits_dev, word_offsets_dev,
                      total_words, E, r, d_in, group, Ut_dev, d_out, X_dev, B, topk_experts_dev,
                      topk_weights_dev, static_cast<int>(k), njobs, nullptr, 0, nullptr, nullptr,
                      nullptr, static_cast<int>(k), Y_dev, stream, reinterpret_cast<char*>(zp),
                      /*timed=*/false);
  // every partial [B k][r] is written by the z kernel before the y kernel
  // reads it, so nothing needs clearing (on the matrix-core path the routing
  // kernel writes the job count and zeroes the rows of unused slots); no
  // events, no library scratch, no copies
  const DecodeGeom g = decode_geometry(njobs, r, d_in, B);
  return decode_launch(g, 1, true, njobs, codes_dev, params_dev, bits_dev, word_offsets_dev,
                       total_words, E, r, d_in, group, Ut_dev, d_out, X_dev, B, nullptr,
                       topk_experts_dev, static_cast<int>(k), topk_weights_dev, nullptr,
                       static_cast<int>(k), zp, Y_dev, static_cast<hipStream_t>(stream),
                       /*timed=*/false);
}

extern "C" bitsmoe_status bitsmoe_moe_decode_in(const uint64_t* codes_dev, const uint16_t* params_dev,
                                                const uint8_t* bits_dev,
                                                const int64_t* word_offsets_dev,
                                                int64_t total_words, int64_t E, int64_t r,
                                                int64_t d_out, int group, const float* Vt_dev,
                                                int64_t d_in, const float* X_dev, int64_t B,
                                                const int64_t* offsets_host,
                                                const int32_t* tokens_host,
                                                const float* weights_host, float* Y_dev,
                                                void* stream) {
  // the units have d_out entries here: the shape rules of the packed rows
  // apply to d_out, the basis rows and tokens have d_in
  bitsmoe_status st = check_decode("moe_decode_in", codes_dev, params_dev, bits_dev,
                                   word_offsets_dev, Vt_dev, X_dev, Y_dev, total_words, E, r, d_out,
                                   group, d_in, B);
  if (st != BITSMOE_OK) return st;
  if (d_in > (1 << 20)) return fail(BITSMOE_ERR_SHAPE, "moe_decode_in: d_in above 2^20");
  RoutingTables rt;
  st = build_routing("moe_decode_in", E, B, offsets_host, tokens_host, weights_host, 4, &rt);
  if (st != BITSMOE_OK) return st;
  int4* jobs_d;
  int64_t* pidx_d;
  float* w_d;
  st = upload_routing("moe_decode_in", rt, weights_host, B, stream, &jobs_d, &pidx_d, &w_d);
  if (st != BITSMOE_OK) return st;
  // segments of 32 outputs: SEGW per workgroup (a power of two up to 256),
  // RSL = 256 / SEGW row slices; rows split over blockIdx.z for about 1024
  // workgroups but at least four rows per thread (each split adds a partial
  // per output to the final sum)
  const int64_t nseg = d_out / kSeg;
  int SEGW = 2;
  while (SEGW < nseg && SEGW < 256) SEGW *= 2;
  const int RSL = 256 / SEGW;
  const int64_t segblocks = (nseg + SEGW - 1) / SEGW;
  int64_t nsplit = std::clamp<int64_t>(1024 / std::max<int64_t>(rt.njobs * segblocks, 1), 1,
                                       std::max<int64_t>(1, (r + 4 * RSL - 1) / (4 * RSL)));
  const int64_t rows_split = (r + nsplit - 1) / nsplit;
  nsplit = (r + rows_split - 1) / rows_split;
  if (nsplit > 65535 || segblocks > 65535) return fail(BITSMOE_ERR_SHAPE, "moe_decode_in: too large");
  // z [B][r], partials yp [nsplit][nnz][d_out]
  const size_t zbytes = (static_cast<size_t>(B * r) * 4 + 255) / 256 * 256;
  char* part = static_cast<char*>(scratch(
      kScratchPart, zbytes + static_cast<size_t>(nsplit * std::max<int64_t>(rt.nnz, 1) * d_out) * 4,
      stream, &st));
  if (!part) return st;
  float* z = reinterpret_cast<float*>(part);
  float* yp = reinterpret_cast<float*>(part + zbytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  {
    KernelTimer timer("moe_decode_in_z", stream);
    hipLaunchKernelGGL(zin_kernel, dim3(static_cast<unsigned>((r + 3) / 4), static_cast<unsigned>(B)),
                       dim3(256), 0, s, Vt_dev, static_cast<int>(r), d_in, X_dev, B, z);
  }
  BITSMOE_LAUNCH_CHECK("moe_decode_in: z launch");
  const uint32_t* pr = reinterpret_cast<const uint32_t*>(params_dev);
  const uint32_t* c32 = reinterpret_cast<const uint32_t*>(codes_dev);
  if (rt.njobs > 0) {
    KernelTimer timer("moe_decode_in_y", stream);
    dim3 grid(static_cast<unsigned>(segblocks), static_cast<unsigned>(rt.njobs),
              static_cast<unsigned>(nsplit));
#define BITSMOE_DECIN(TT)                                                                           \
  hipLaunchKernelGGL(yin_kernel<TT>, grid, dim3(256), 0, s, c32, pr, bits_dev, word_offsets_dev,    \
                     total_words, static_cast<int>(r), static_cast<int>(d_out), group, SEGW,        \
                     static_cast<int>(rows_split), z, jobs_d, w_d, rt.nnz, yp)
    if (rt.T == 4) BITSMOE_DECIN(4); else BITSMOE_DECIN(1);
#undef BITSMOE_DECIN
  }
  BITSMOE_LAUNCH_CHECK("moe_decode_in: y launch");
  {
    KernelTimer timer("moe_decode_in_sum", stream);
    hipLaunchKernelGGL(ysum_kernel, dim3(static_cast<unsigned>((d_out + 63) / 64), static_cast<unsigned>(B)),
                       dim3(256), 0, s, yp, static_cast<int>(nsplit), rt.nnz, pidx_d,
                       static_cast<int>(rt.kmax), d_out, B, Y_dev);
  }
  BITSMOE_LAUNCH_CHECK("moe_decode_in: sum launch");
  return ok();
}
