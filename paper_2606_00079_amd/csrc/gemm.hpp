// bf16 matrix-core ("NT") GEMM engine for gfx950.
//
// Every contraction of the quantizer has the form
//     acc[i][j] = sum_k A[i][k] * B[j][k]
// with both operands stored as bf16 rows that are contiguous along k: the
// calibration Gram (A = B = X^T), the cross-expert Gram (A = B = the expert
// rows, k running over experts and input channels), the spectral factors
// (A = U^T, B = W_e^T) and the loss table (A = off-diagonal H, B = error
// rows).  What happens to the fp32 accumulators is left to an epilogue
// functor.
//
// Kernel shape: a BM x BN workgroup tile, 4 waves of 64 lanes in a 2 x 2
// grid, each wave owning a (BM/2) x (BN/2) block of v_mfma_f32_32x32x16_bf16
// (or _f16 when the operands are fp16)
// accumulators.  K advances 32 at a time through four LDS stages filled by
// direct global->LDS loads (global_load_lds_dwordx4): while K tile i is
// multiplied, tile i+3 is loaded into the buffer tile i-1 used.  One wave
// per SIMD issues in order, so the loads of a refill and the fragment reads
// of the next K=16 step are interleaved one per matrix-core op and spread
// over both steps of the tile (see `mfmas`); waits are explicit s_waitcnt
// counts and barriers bare s_barrier.  LDS rows are 64 bytes and the four
// 16-byte chunks of row r are stored XOR-swizzled by (r / 4) mod 4, so the
// fragment reads of the matrix-core operands are free of bank conflicts.
//
// The K index is a flattened (pass, segment, k) triple:
//   * passes   let one launch add up to 4 products A_p B_p^T into the same
//              accumulators (used for hi/lo bf16 splits of fp32 data);
//   * segments let K run over several equally long pieces that are a fixed
//              stride apart in memory (the experts of W for M = sum W_e W_e^T).
// gridDim.y splits K (split-K); gridDim.z is a batch index with its own
// operand strides.
//
// Tile order.  Workgroups are dispatched round-robin over the 8 XCDs, each
// with its own L2.  The linear workgroup id is first remapped so that every
// XCD receives a contiguous range of logical ids, and logical ids walk the
// tiles in groups of `group_n` column tiles, rows fastest: the workgroups
// resident on one XCD then share both their A row-slabs and B column-slabs
// through that XCD's L2.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace bitsmoe {
namespace gemm {

constexpr int BK = 32;             // unit in which Problem::ktiles counts K
constexpr int kKAlign = 64;        // every K segment (Problem::kseg) is a multiple of this
constexpr int kThreads = 256;
// Matrix-core ops between the LDS read of a bf16 B fragment and its widening
// (each op runs 32 cycles: about the LDS read's latency under load at four;
// two to six measured the same).
constexpr int kCvtLag = 4;

// Compile-time loop: calls f(std::integral_constant<int, I>) for I = 0..N-1.
template <int I, int N>
struct StaticFor {
  template <class Fn>
  __device__ __forceinline__ static void run(Fn&& fn) {
    fn(std::integral_constant<int, I>());
    StaticFor<I + 1, N>::run(fn);
  }
};
template <int N>
struct StaticFor<N, N> {
  template <class Fn>
  __device__ __forceinline__ static void run(Fn&&) {}
};
// A compile-time range [A, B) of a refill's direct loads.
template <int A, int B>
struct LoadRange {
  static constexpr int first = A, second = B;
};
constexpr int kXcds = 8;

// Operand layouts.  Row-major (kstep == 0): row r, column k at r * ld + k;
// rows past `rows` are clamped to the last row.  K-tiled (kstep != 0, for a
// kernel with BK-wide K steps and tiles of T rows on this side): the T x BK
// block of row tile t and K tile q is contiguous, at t * rtile + q * kstep
// (kstep = T * BK), rows BK elements apart inside it; every row tile is
// allocated in full, so nothing is clamped.  A K step then reads whole cache
// lines instead of 64-byte halves of them.  K-major ("KN", B side only, with
// the kernel's BKN flag): element (k, n) at k * ld + n, i.e. K runs over
// rows; kstep = BK * ld, rtile = BN, columns past `rows` are clamped.  The
// B fragments are then read from LDS with the 16-bit transposing read.
constexpr int kTileK = 32;  // K width of a K-tiled block (must equal the kernel's K step)
struct Side {
  const uint16_t* pass[4];  // base pointer of each pass
  int64_t ld;               // row-major: elements between consecutive rows
  int64_t estride;          // elements between consecutive K segments
  int64_t bstride;          // elements between batches (blockIdx.z)
  int64_t rows;             // row-major: valid rows
  int64_t kstep;            // K-tiled: elements between consecutive K tiles (0 = row-major)
  int64_t rtile;            // K-tiled: elements between consecutive row tiles
  int repeat_k;             // 1: every K tile of a segment starts at the segment's
                            // base (the side's tile is reused; estride advances)
};

// Element offset of (r, k) in a K-tiled matrix of K columns with T-row tiles.
__host__ __device__ __forceinline__ int64_t tiled_offset(int64_t r, int64_t k, int64_t K, int T) {
  return ((r / T) * (K / kTileK) + k / kTileK) * (static_cast<int64_t>(T) * kTileK) +
         (r % T) * kTileK + (k % kTileK);
}

struct Problem {
  Side a, b;
  int passes;
  int segs;          // K segments per pass
  int64_t kseg;      // K elements per segment (multiple of BK)
  int64_t ktiles;    // passes * segs * kseg / BK
  int splits;        // gridDim.y
  int tiles_m, tiles_n;
  int symmetric;     // 1: only tiles with tm <= tn are launched (gridDim.x = T(T+1)/2)
  int group_n;       // column tiles per ordering group (non-symmetric; paired: per
                     // group_n column tiles, all pairs of each)
  int64_t a_batch_rows;  // paired only: if > 0, the A operand of column tile tn is
                         // batch (tn * BN) / a_batch_rows (stride a.bstride): one A per
                         // block of B rows (a multiple of BN)
  // run_if: when not null, every workgroup returns at once unless *run_if is
  // nonzero (a launch made conditional on an earlier launch's flag)
  const int* run_if;
  // flat > 0 (not paired): one-dimensional grid of batches x splits x flat
  // tiles (flat = the tiles of one batch and split), blockIdx.y = .z = 0.
  // The linear id is XCD-remapped first, so the tiles of one split of one
  // batch (which read the same K slice of the same operands) run on one XCD
  // and share its L2.
  int flat;
  // persist > 0 (with flat, not paired): the same persist = batches x splits
  // x flat logical tiles, walked by a grid of fewer workgroups (a multiple
  // of the XCD count): XCD x takes the same contiguous range of logical ids
  // as in the flat launch, and its workgroups take them in turn.  With an
  // epilogue that leaves the LDS alone, each workgroup issues the first K
  // tiles of its next tile before the epilogue of the current one, so the
  // epilogue's stores overlap the next tile's loads.
  int64_t persist;
};

// Logical (XCD-contiguous) range of XCD x when n logical ids are spread as
// xcd_remap spreads them: [*start, *start + *len).
__host__ __device__ __forceinline__ void xcd_range(int64_t n, int x, int64_t* start, int64_t* len) {
  const int64_t q = n / kXcds, rem = n % kXcds;
  *start = x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q;
  *len = q + (x < rem ? 1 : 0);
}

// XCD-contiguous logical id of the linear workgroup id t (of n in total).
__device__ __forceinline__ int xcd_remap(int t, int n) {
  const int x = t % kXcds, i = t / kXcds;
  const int q = n / kXcds, rem = n % kXcds;
  return (x < rem) ? x * (q + 1) + i : rem * (q + 1) + (x - rem) * q + i;
}

// Tile of logical (XCD-remapped) id t.
__device__ __forceinline__ void tile_coords_logical(const Problem& p, int t, int* tm, int* tn) {
  if (p.symmetric) {
    int r = 0;
    while (t >= p.tiles_m - r) {
      t -= p.tiles_m - r;
      ++r;
    }
    *tm = r;
    *tn = r + t;
    return;
  }
  const int per_group = p.group_n * p.tiles_m;
  const int g = t / per_group, w = t - g * per_group;
  const int first_n = g * p.group_n;
  // the grid holds tiles_m * tiles_n workgroups, so the last (possibly
  // narrower) group still has w / tiles_m < its width
  *tm = w % p.tiles_m;
  *tn = first_n + w / p.tiles_m;
}
__device__ __forceinline__ void tile_coords(const Problem& p, int t, int n, int* tm, int* tn) {
  tile_coords_logical(p, xcd_remap(t, n), tm, tn);
}

// Paired upper-triangle schedule (for a symmetric form: A is the square
// d x d operand, one pass, one segment, no split-K, BM-wide K blocks).  Row
// tile tm needs only the K blocks at and right of its diagonal block
// (tiles_m - tm of them), so every workgroup runs two jobs of tiles_m + 1
// blocks in all: row tiles tm and tiles_m - 1 - tm of one column tile, or,
// for an odd tiles_m, the middle row tile of two neighbouring column tiles.
// Jobs are counted in units of one column tile (even tiles_m, tiles_m / 2
// workgroups each) or two (odd, tiles_m workgroups each); group_n units
// form an ordering group, workgroups of a unit consecutive.
__host__ __device__ __forceinline__ int64_t paired_workgroups(int tiles_m, int64_t tiles_n) {
  return (tiles_m % 2 == 0) ? tiles_n * (tiles_m / 2) : (tiles_n + 1) / 2 * tiles_m;
}
__host__ __device__ __forceinline__ int paired_unit_workgroups(int tiles_m) {
  return (tiles_m % 2 == 0) ? tiles_m / 2 : tiles_m;
}
// Jobs (tm0, tn0) then (tm1, tn1) of workgroup t (of n); returns how many
// exist (0, 1 or 2: the second column tile of the last unit may be missing).
__device__ __forceinline__ int paired_jobs(const Problem& p, int t, int n, int* tm0, int* tn0,
                                           int* tm1, int* tn1) {
  const int T = p.tiles_m;
  const int per_unit = paired_unit_workgroups(T);
  t = xcd_remap(t, n);
  const int per_group = p.group_n * per_unit;
  const int g = t / per_group, w = t - g * per_group;
  const int unit = g * p.group_n + w / per_unit, s = w % per_unit;
  if (T % 2 == 0) {
    *tm0 = s;
    *tm1 = T - 1 - s;
    *tn0 = *tn1 = unit;
    return 2;
  }
  const int h = (T - 1) / 2;  // pairs per column tile; the middle row tile is h
  if (s < T - 1) {
    const int tn = 2 * unit + s / h;
    *tm0 = s % h;
    *tm1 = T - 1 - s % h;
    *tn0 = *tn1 = tn;
    return tn < p.tiles_n ? 2 : 0;
  }
  *tm0 = *tm1 = h;
  *tn0 = 2 * unit;
  *tn1 = 2 * unit + 1;
  return *tn1 < p.tiles_n ? 2 : 1;
}

// v made wave-uniform (held in scalar registers from here on).
__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const uint64_t u = static_cast<uint64_t>(v);
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u)));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32)));
  return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}
__device__ __forceinline__ int uniform32(int v) { return __builtin_amdgcn_readfirstlane(v); }

// The pass bases of one side for batch z and first tile row row0, as a
// shift register: q0 is the current pass, and moving to the next pass shifts
// the others down by selects (indexing the bases by pass number would turn
// them into a memory table).
struct PassBases {
  const uint16_t* q0;
  const uint16_t* q1;
  const uint16_t* q2;
  const uint16_t* q3;
  __device__ __forceinline__ void init(const Side& s, int64_t z, int64_t tile, int rows_per_tile) {
    const int64_t off = z * s.bstride + (s.kstep != 0 ? tile * s.rtile : tile * rows_per_tile * s.ld);
    q0 = s.pass[0] + off;
    q1 = s.pass[1] + off;
    q2 = s.pass[2] + off;
    q3 = s.pass[3] + off;
  }
  __device__ __forceinline__ void advance(bool w) {
    q0 = w ? q1 : q0;
    q1 = w ? q2 : q1;
    q2 = w ? q3 : q2;
  }
  __device__ __forceinline__ void make_uniform() {
    auto u = [](const uint16_t* ptr) {
      return reinterpret_cast<const uint16_t*>(uniform64(reinterpret_cast<int64_t>(ptr)));
    };
    q0 = u(q0);
    q1 = u(q1);
    q2 = u(q2);
    q3 = u(q3);
  }
};

// Position of a K tile in the flattened (pass, segment, k) index: the base
// of its pass and its element offset from that base on each side.  Advanced
// by scalar selects inside the K loop (no division, branch or memory load).
template <int KB>
struct KPos {
  int64_t seg, k0;
  int64_t offa, offb;    // element offsets of the tile from the pass bases
  int64_t stepa, stepb;  // per K tile
  int64_t jumpa, jumpb;  // extra at a segment boundary
  PassBases ba, bb;
  __device__ __forceinline__ void init(const Problem& p, int64_t kt, int64_t z, int tm, int tn,
                                       int BM, int BN) {
    const int64_t tiles_seg = p.kseg / KB;
    const int64_t per_pass = static_cast<int64_t>(p.segs) * tiles_seg;
    const int pass = static_cast<int>(kt / per_pass);
    const int64_t rem = kt - static_cast<int64_t>(pass) * per_pass;
    seg = rem / tiles_seg;
    const int64_t ki = rem - seg * tiles_seg;  // K tile within the segment
    k0 = ki * KB;
    ba.init(p.a, z, tm, BM);
    bb.init(p.b, z, tn, BN);
    for (int q = 0; q < pass; ++q) {
      ba.advance(true);
      bb.advance(true);
    }
    ba.make_uniform();
    bb.make_uniform();
    stepa = uniform64(p.a.repeat_k ? 0 : (p.a.kstep != 0 ? p.a.kstep : KB));
    stepb = uniform64(p.b.repeat_k ? 0 : (p.b.kstep != 0 ? p.b.kstep : KB));
    jumpa = uniform64(p.a.estride - tiles_seg * stepa);
    jumpb = uniform64(p.b.estride - tiles_seg * stepb);
    seg = uniform64(seg);
    k0 = uniform64(k0);
    offa = uniform64(seg * p.a.estride + ki * stepa);
    offb = uniform64(seg * p.b.estride + ki * stepb);
  }
  __device__ __forceinline__ const uint16_t* a_ptr() const { return ba.q0 + offa; }
  __device__ __forceinline__ const uint16_t* b_ptr() const { return bb.q0 + offb; }
  __device__ __forceinline__ void next(const Problem& p) {
    k0 += KB;
    offa += stepa;
    offb += stepb;
    const bool wrap = k0 == p.kseg;
    k0 = wrap ? 0 : k0;
    offa = wrap ? offa + jumpa : offa;
    offb = wrap ? offb + jumpb : offb;
    seg += wrap ? 1 : 0;
    const bool wrap2 = seg == p.segs;
    seg = wrap2 ? 0 : seg;
    offa = wrap2 ? 0 : offa;
    offb = wrap2 ? 0 : offb;
    ba.advance(wrap2);
    bb.advance(wrap2);
  }
};

// K walk of a one-pass, one-segment problem (persistent launches): the
// position of K tile kt is kt steps from the tile's base on each side.
template <int KB>
struct KPos1 {
  const uint16_t* ba;
  const uint16_t* bb;
  int64_t offa, offb, stepa, stepb;
  __device__ __forceinline__ void init(const Problem& p, int64_t kt, int64_t z, int tm, int tn,
                                       int BM, int BN) {
    PassBases a, b;
    a.init(p.a, z, tm, BM);
    b.init(p.b, z, tn, BN);
    ba = reinterpret_cast<const uint16_t*>(uniform64(reinterpret_cast<int64_t>(a.q0)));
    bb = reinterpret_cast<const uint16_t*>(uniform64(reinterpret_cast<int64_t>(b.q0)));
    stepa = uniform64(p.a.kstep != 0 ? p.a.kstep : KB);
    stepb = uniform64(p.b.kstep != 0 ? p.b.kstep : KB);
    offa = uniform64(kt * stepa);
    offb = uniform64(kt * stepb);
  }
  __device__ __forceinline__ const uint16_t* a_ptr() const { return ba + offa; }
  __device__ __forceinline__ const uint16_t* b_ptr() const { return bb + offb; }
  __device__ __forceinline__ void next(const Problem&) {
    offa += stepa;
    offb += stepb;
  }
};

// K walk of one job of the paired-triangle schedule (one pass, one segment,
// no split-K): K tiles q0, q0 + 1, ... (or q0, q0 - 1, ...) for `turn`
// visits, then from tile qt downwards.  Scalar selects only; offsets within a
// row tile are 32-bit (the caller keeps ktiles * kstep below 2^31).
template <int KB>
struct TriWalk {
  const uint16_t* ba;
  const uint16_t* bb;
  int offa, offb;    // element offsets of the current tile from the tile bases
  int stepa, stepb;  // signed, per K tile
  int n, turn;       // visits so far; the visit at which the walk turns (-1: never)
  int toffa, toffb;  // offsets of tile qt
  __device__ __forceinline__ void init(const Problem& p, int64_t z, int tm, int tn, int BM, int BN,
                                       int64_t q0, bool up, int64_t turn_at, int64_t qt) {
    PassBases a, b;
    const int64_t za = p.a_batch_rows > 0 ? static_cast<int64_t>(tn) * BN / p.a_batch_rows : z;
    a.init(p.a, za, tm, BM);
    b.init(p.b, z, tn, BN);
    ba = reinterpret_cast<const uint16_t*>(uniform64(reinterpret_cast<int64_t>(a.q0)));
    bb = reinterpret_cast<const uint16_t*>(uniform64(reinterpret_cast<int64_t>(b.q0)));
    const int sa = static_cast<int>(p.a.kstep != 0 ? p.a.kstep : KB);
    const int sb = static_cast<int>(p.b.kstep != 0 ? p.b.kstep : KB);
    offa = uniform32(static_cast<int>(q0) * sa);
    offb = uniform32(static_cast<int>(q0) * sb);
    stepa = uniform32(up ? sa : -sa);
    stepb = uniform32(up ? sb : -sb);
    n = 0;
    turn = uniform32(static_cast<int>(turn_at));
    toffa = uniform32(static_cast<int>(qt) * sa);
    toffb = uniform32(static_cast<int>(qt) * sb);
  }
  __device__ __forceinline__ void next() {
    ++n;
    offa += stepa;
    offb += stepb;
    const bool t = n == turn;
    offa = t ? toffa : offa;
    offb = t ? toffb : offb;
    stepa = t ? -stepa : stepa;
    stepb = t ? -stepb : stepb;
  }
};

// One wave-wide direct global->LDS load of 16 bytes per lane: lane l reads
// base + voff_l bytes and its 16 bytes land at LDS byte address lds + 16 l.
// `base` and `lds` are wave-uniform.  Issued through inline assembly so that
// the compiler neither tracks the LDS write nor inserts waits for it: every
// caller waits explicitly (s_waitcnt vmcnt) and synchronizes the workgroup
// before the data is read.  M0 carries the LDS address; nothing else in the
// kernels that use this helper uses M0.
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, const void* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds)));
  // readfirstlane returns a signed int: both halves are zero-extended
  // explicitly, or a low word with bit 31 set would smear into the high word.
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32)));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b)));
  const uint64_t bu = (static_cast<uint64_t>(hi) << 32) | static_cast<uint64_t>(lo);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(bu), "s"(l)
               : "memory");
}

// Swizzle: the LDS serves a 16-byte read for 16 lanes per cycle out of 64
// four-byte banks (256 bytes), so with KB-element rows (KB/8 chunks) chunk j
// of row r is stored in slot j ^ ((r / (16 / (KB/8))) mod (KB/8)): sixteen
// consecutive rows read at the same chunk then cover all 64 banks once
// (KB = 64: key (r/2) mod 8; KB = 32: key (r/4) mod 4).
template <int KB>
__device__ __forceinline__ int swz(int r, int j) {
  constexpr int KC = KB / 8;
  return j ^ ((r / (16 / KC)) & (KC - 1));
}
// LDS element offset of chunk j (8 bf16) of row r.
template <int KB>
__device__ __forceinline__ int lds_off(int r, int j) { return r * KB + (swz<KB>(r, j) << 3); }

// s_waitcnt on the vector-memory counter only (expcnt and lgkmcnt left at
// their maxima), in the gfx9 encoding: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in
// bits 15:14.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// The same, and every LDS read of this wave returned (lgkmcnt 0).
template <int N>
__device__ __forceinline__ void wait_vmcnt_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// The K-loop stage buffers, free once the loop is done; epilogues may use
// them as scratch: kStages A buffers then kStages B buffers.
struct StageLds {
  uint16_t* a;        // A stage buffers, a_elems bf16 in all, contiguous
  uint16_t* b;        // B stage buffers, b_elems bf16 in all, contiguous
  int a_elems, b_elems;
  // K tiles this workgroup visited; the n-th visited tile (n = 0, 1, ...)
  // was staged in buffer n % stages, so the last `stages` of them are still
  // there (in the swizzled stage layout)
  int64_t nk;
  int stages;
  // 16 KiB piece k of the A buffers followed by the B buffers
  __device__ __forceinline__ uint16_t* piece(int k) const {
    const int per_a = a_elems / 8192;
    return k < per_a ? a + k * 8192 : b + (k - per_a) * 8192;
  }
};

// Accumulator fragment bookkeeping handed to epilogues: the four waves as
// NWM x NWN, wave (wm, wn) owning rows wm * WM .. and columns wn * WN .. of
// the tile.
template <int BM, int BN, int NWM = 2, int NWN = 2>
struct Frag {
  static_assert(NWM * NWN == 4, "four waves");
  static constexpr int WM = BM / NWM, WN = BN / NWN;
  static constexpr int FM = WM / 32;
  static constexpr int FN = WN / 32;
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

// For epilogues that store rows: lane k of each group of four lanes holds rows R .. R+3 of column c0 + k
// on entry and row R + k of columns c0 .. c0+3 on exit (a 4 x 4 transpose
// by two butterfly exchanges with DPP quad permutations).
template <int CTRL>
__device__ __forceinline__ float quad_dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ void quad_transpose(float (&a)[4], int k) {
  constexpr int kSwap1 = 0xB1;  // quad_perm [1, 0, 3, 2]: lane k ^ 1
  constexpr int kSwap2 = 0x4E;  // quad_perm [2, 3, 0, 1]: lane k ^ 2
  const bool o1 = (k & 1) != 0;
  float s0 = quad_dpp<kSwap1>(o1 ? a[0] : a[1]);
  float s1 = quad_dpp<kSwap1>(o1 ? a[2] : a[3]);
  a[0] = o1 ? s0 : a[0];
  a[1] = o1 ? a[1] : s0;
  a[2] = o1 ? s1 : a[2];
  a[3] = o1 ? a[3] : s1;
  const bool o2 = (k & 2) != 0;
  s0 = quad_dpp<kSwap2>(o2 ? a[0] : a[2]);
  s1 = quad_dpp<kSwap2>(o2 ? a[1] : a[3]);
  a[0] = o2 ? s0 : a[0];
  a[1] = o2 ? s1 : a[1];
  a[2] = o2 ? a[2] : s0;
  a[3] = o2 ? a[3] : s1;
}

// 16-bit operand element: bf16 (default) or fp16.
template <bool F16>
struct Operand {
  typedef bf16x8 vec;
  static __device__ __forceinline__ f32x16 mfma(vec a, vec b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Operand<true> {
  typedef f16x8 vec;
  static __device__ __forceinline__ f32x16 mfma(vec a, vec b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};

// Transposing 16-bit LDS read: within each group of 16 lanes, lane j gets
// element (j mod 4) of the 8-byte run addressed by lane 4 q + j / 4 as its
// element q.  So if lane s of a group points at row k + s / 4, columns
// c + 4 (s mod 4) .. + 3 of a row-major [K][N] tile, lane j receives rows
// k .. k + 3 of column c + j.
typedef short __attribute__((ext_vector_type(4))) s16x4;
__device__ __forceinline__ s16x4 ds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(reinterpret_cast<uintptr_t>(p)));
}

// KN stage layout: BK rows of BN entries (512-byte rows for BN = 256), the
// 16-byte chunk c of row r stored at chunk c ^ (4 (r mod 4)): one half-wave
// of transposing reads (4 rows x 4 chunks x 2 halves) covers all 64 banks.
__device__ __forceinline__ int kn_swz(int r, int c) { return c ^ (4 * (r & 3)); }

// Eight bf16 values (bit patterns, two per dword) -> eight fp16 values: each
// bf16 is widened to the fp32 of the same value (its bits in the upper
// half) and rounded to fp16 to nearest even, two at a time.  bf16 values
// of magnitude 2^-14 .. 65504 convert exactly (fp16 has the wider
// significand), 2^-17 .. 2^-14 land exactly on fp16 subnormals, smaller ones
// round on the 2^-24 grid, larger ones become infinite.
__device__ __forceinline__ f16x8 bf16x8_to_f16x8(const uint32_t (&w)[4]) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  h2 o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = __uint_as_float(w[i] << 16);
    const float hi = __uint_as_float(w[i] & 0xffff0000u);
    o[i] = h2{static_cast<_Float16>(lo), static_cast<_Float16>(hi)};
  }
  return f16x8{o[0].x, o[0].y, o[1].x, o[1].y, o[2].x, o[2].y, o[3].x, o[3].y};
}

// CVTB: the B operand is bf16 in memory and is multiplied as fp16 (F16):
// each B fragment is converted in registers after its LDS read.
// PERSIST: compiled for a persistent launch (Problem::persist > 0).
// ONEK: compiled for a one-pass, one-segment problem without repeat_k (the
// K walk is a fixed step per tile; persistent launches always are).
template <int BM, int BN, int KB, int STAGES, class Epi, bool F16 = false, bool BKN = false,
          bool PAIRED = false, bool CVTB = false, bool PERSIST = false, bool ONEK = false,
          int NWN = 2>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_nt_kernel(Problem p, Epi epi) {
  static_assert(BM % 64 == 0 && BN % 64 == 0, "tile");
  static_assert(!CVTB || F16, "converted B fragments are fp16");
  static_assert(!PERSIST || (!PAIRED && !Epi::kUsesLds), "persistent: one tile per job, LDS-free epilogue");
  static_assert(!ONEK || !PAIRED, "the paired schedule has its own K walk");
  // (persistent: p.passes == 1 and p.segs == 1, see KPos1)
  if (p.run_if && *p.run_if == 0) return;  // whole workgroup
  static_assert(!BKN || (BN == 256 && KB == 32), "KN B operand: 256-wide N tiles, 32-wide K steps");
  static_assert(KB == 32 || KB == 64, "K step");
  static_assert(STAGES >= 2 && STAGES <= 6, "stages");
  constexpr int KC = KB / 8;        // 16-byte chunks per LDS row
  constexpr int RPB = 512 / KB;     // rows per 1 KiB block (one wave-wide direct load)
  constexpr int AW = BM / RPB / 4;  // direct 1 KiB loads per wave per stage
  constexpr int BW = BN / RPB / 4;
  constexpr int LPS = AW + BW;      // vector-memory instructions per wave per stage
  constexpr int ASZ = BM * KB, BSZ = BN * KB;  // elements per stage
  static_assert(AW >= 1 && BW >= 1, "tile too small");
  // NWN = 4 (waves side by side along N, each all BM rows): every B fragment
  // is read, and with CVTB widened, by one wave instead of two
  using F = Frag<BM, BN, 4 / NWN, NWN>;
  static_assert(F::WM % 32 == 0 && F::WN % 32 == 0, "32 x 32 fragments per wave");

  __shared__ __align__(1024) uint16_t As[STAGES * ASZ];
  __shared__ __align__(1024) uint16_t Bs[STAGES * BSZ];

  const int tid = threadIdx.x;
  F f;
  f.lane = tid & 63;
  // wave-uniform: keeps everything derived from it in scalar registers
  f.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  f.wm = f.wave / NWN;
  f.wn = f.wave % NWN;
  // PAIRED: gridDim.x = paired_workgroups(tiles_m, tiles_n), two jobs each
  // (see paired_jobs); persistent: the logical tiles pjob0 + j pstride;
  // otherwise one tile per workgroup.
  int njobs = 1, tm0 = 0, tn0 = 0, tm1 = 0, tn1 = 0;
  int64_t pjob0 = 0, pstride = 0;
  // logical id L of a flat or persistent launch -> tile, batch and split
  auto flat_coords = [&](int64_t L, int* tm, int* tn, int64_t* z, int* ks) {
    const int64_t per_z = static_cast<int64_t>(p.splits) * p.flat;
    const int64_t zz = L / per_z;
    const int rem = static_cast<int>(L - zz * per_z);
    *z = zz;
    *ks = rem / p.flat;
    tile_coords_logical(p, rem - *ks * p.flat, tm, tn);
  };
  if constexpr (PAIRED) {
    njobs = paired_jobs(p, blockIdx.x, gridDim.x, &tm0, &tn0, &tm1, &tn1);
    if (njobs == 0) return;  // whole workgroup: past the last column tile
    f.ks = blockIdx.y;
    f.z = blockIdx.z;
  } else if (PERSIST) {
    const int x = static_cast<int>(blockIdx.x % kXcds), wi = static_cast<int>(blockIdx.x / kXcds);
    const int wx = static_cast<int>(gridDim.x / kXcds) + (x < static_cast<int>(gridDim.x % kXcds) ? 1 : 0);
    int64_t start, len;
    xcd_range(p.persist, x, &start, &len);
    if (wi >= len) return;  // whole workgroup: nothing left on its XCD
    njobs = static_cast<int>((len - wi + wx - 1) / wx);
    pjob0 = start + wi;
    pstride = wx;
    flat_coords(pjob0, &tm0, &tn0, &f.z, &f.ks);
  } else if (p.flat > 0) {
    flat_coords(xcd_remap(blockIdx.x, gridDim.x), &tm0, &tn0, &f.z, &f.ks);
  } else {
    tile_coords(p, blockIdx.x, gridDim.x, &tm0, &tn0);
    f.ks = blockIdx.y;
    f.z = blockIdx.z;
  }
  f.tm = tm0;
  f.tn = tn0;

  const int64_t ktiles = p.ktiles * BK / KB;  // K tiles of this kernel's step
  int64_t kt0 = ktiles * f.ks / p.splits;
  int64_t kt1 = ktiles * (f.ks + 1) / p.splits;

  // Direct global->LDS loads.  Wave instruction i of this wave fills the
  // 1 KiB LDS block b = wave + 4 i (rows b*RPB .. b*RPB+RPB-1); lane l lands
  // at byte 16 l of the block, i.e. row b*RPB + l/KC, slot l%KC, so it fetches
  // the global chunk that the swizzle stores in that slot.  Rows past the end
  // are clamped to the last row: their accumulators are never stored.
  uint32_t oa[AW], ob[BW];  // byte offsets from the tile's first element
  const bool a_tiled = p.a.kstep != 0, b_tiled = p.b.kstep != 0;
  auto set_offsets = [&](int tm, int tn) {
  const int64_t a_row0 = static_cast<int64_t>(tm) * BM;
  const int64_t b_row0 = static_cast<int64_t>(tn) * BN;
#pragma unroll
  for (int i = 0; i < AW; ++i) {
    const int r = (f.wave + 4 * i) * RPB + f.lane / KC;
    const int j = swz<KB>(r, f.lane % KC);
    const int64_t gr = (a_row0 + r < p.a.rows) ? a_row0 + r : p.a.rows - 1;
    oa[i] = a_tiled ? static_cast<uint32_t>((r * KB + 8 * j) * 2)
                    : static_cast<uint32_t>(((gr - a_row0) * p.a.ld + 8 * j) * 2);
  }
#pragma unroll
  for (int i = 0; i < BW; ++i) {
    if constexpr (BKN) {
      // 1 KiB block b = rows 2b, 2b+1 (K) of the tile, 512 bytes (N) each;
      // chunks past column `rows` are clamped to the last full chunk
      const int r = 2 * (f.wave + 4 * i) + f.lane / 32;
      const int c = kn_swz(r, f.lane % 32);
      int64_t col = b_row0 + 8 * c;
      col = col + 8 <= p.b.rows ? col : p.b.rows - 8;
      ob[i] = static_cast<uint32_t>((r * p.b.ld + (col - b_row0)) * 2);
    } else {
      const int r = (f.wave + 4 * i) * RPB + f.lane / KC;
      const int j = swz<KB>(r, f.lane % KC);
      const int64_t gr = (b_row0 + r < p.b.rows) ? b_row0 + r : p.b.rows - 1;
      ob[i] = b_tiled ? static_cast<uint32_t>((r * KB + 8 * j) * 2)
                      : static_cast<uint32_t>(((gr - b_row0) * p.b.ld + 8 * j) * 2);
    }
  }
  };
  // persistent launches walk a one-pass, one-segment K (checked by the host)
  std::conditional_t<PERSIST || ONEK, KPos1<KB>, KPos<KB>> kp;
  TriWalk<KB> tw;
  // Loads of the next K tile into stage buffer s, one wave instruction at a
  // time (q < LPS) so that they can be spread between matrix-core ops.
  struct Issue {
    const uint16_t* pa;
    const uint16_t* pb;
    int s;
  };
  auto issue_begin = [&](int s) {
    if constexpr (PAIRED) {
      Issue is{tw.ba + tw.offa, tw.bb + tw.offb, s};
      tw.next();
      return is;
    } else {
      Issue is{kp.a_ptr(), kp.b_ptr(), s};
      kp.next(p);
      return is;
    }
  };
  auto issue_part = [&](const Issue& is, int q) {
    if (q < AW)
      dma16(is.pa, oa[q], As + is.s * ASZ + (f.wave + 4 * q) * (RPB * KB));
    else
      dma16(is.pb, ob[q - AW], Bs + is.s * BSZ + (f.wave + 4 * (q - AW)) * (RPB * KB));
  };
  auto issue = [&](int s) {
    const Issue is = issue_begin(s);
#pragma unroll
    for (int q = 0; q < LPS; ++q) issue_part(is, q);
  };

  const int arow = f.wm * F::WM + (f.lane & 31);
  const int brow = f.wn * F::WN + (f.lane & 31);
  const int jq = f.lane >> 5;
  // Two register sets of operand fragments: while the matrix cores work on
  // one K=16 step, the fragments of the next step are read into the other.
  using Op = Operand<F16>;
  typename Op::vec fa[2][F::FM], fb[2][F::FN];
  // CVTB: the raw bf16 B fragments of the step being read; each is widened
  // into fb a few matrix-core ops after its read (cvt_frag), once the read
  // has returned, so that the wave does not wait on the LDS.
  uint32_t rawb[CVTB ? F::FN : 1][4];
  // Operand fragment q of the K=16 step kk of stage s into register set
  // `set`, in the order the matrix-core ops of a step first use them: A0,
  // then B0 .. B(FN-1), then A1 .. A(FM-1).
  auto read_frag = [&](auto set, auto qq, int s, int kk) {
    constexpr int T = decltype(set)::value;
    constexpr int q = decltype(qq)::value;
    const int j = 2 * kk + jq;
    if constexpr (q == 0 || q > F::FN) {
      constexpr int mi = q == 0 ? 0 : q - F::FN;
      const uint16_t* la = As + s * ASZ;
      fa[T][mi] = *reinterpret_cast<const typename Op::vec*>(&la[lds_off<KB>(arow + 32 * mi, j)]);
    } else {
      constexpr int ni = q - 1;
      const uint16_t* lb = Bs + s * BSZ;
      if constexpr (BKN) {
        // rows 16 kk + 8 (lane / 32) + 4 t + (lane % 16) / 4, column
        // n + 16 ((lane / 16) % 2) + 4 (lane % 4) of the [32][256] stage tile
        const int col = f.wn * F::WN + 32 * ni + 16 * ((f.lane >> 4) & 1) + 4 * (f.lane & 3);
        s16x4 h[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int r = 16 * kk + 8 * jq + 4 * t + ((f.lane & 15) >> 2);
          h[t] = ds_read_tr16(lb + r * BN + (kn_swz(r, col >> 3) << 3) + (col & 7));
        }
        if constexpr (CVTB) {
          __builtin_memcpy(rawb[ni], &h[0], 8);
          __builtin_memcpy(rawb[ni] + 2, &h[1], 8);
        } else {
          fb[T][ni] = __builtin_bit_cast(typename Op::vec,
                                         __builtin_shufflevector(h[0], h[1], 0, 1, 2, 3, 4, 5, 6, 7));
        }
      } else if constexpr (CVTB) {
        const uint4 v = *reinterpret_cast<const uint4*>(&lb[lds_off<KB>(brow + 32 * ni, j)]);
        rawb[ni][0] = v.x;
        rawb[ni][1] = v.y;
        rawb[ni][2] = v.z;
        rawb[ni][3] = v.w;
      } else {
        fb[T][ni] = *reinterpret_cast<const typename Op::vec*>(&lb[lds_off<KB>(brow + 32 * ni, j)]);
      }
    }
  };
  auto cvt_frag = [&](auto set, auto nn) {
    constexpr int T = decltype(set)::value;
    constexpr int ni = decltype(nn)::value;
    if constexpr (CVTB) fb[T][ni] = bf16x8_to_f16x8(rawb[ni]);
  };
  constexpr int NFR = F::FM + F::FN;  // fragment reads per step
  auto read_frags = [&](auto set, int s, int kk) {
    StaticFor<0, NFR>::run([&](auto qq) { read_frag(set, qq, s, kk); });
    StaticFor<0, F::FN>::run([&](auto nn) { cvt_frag(set, nn); });
  };
  // The matrix-core ops of one K=16 step from fragment set `set`.  Between
  // them go the other instructions of the step: the NFR fragment reads of
  // the next step into the other set (`frs`: stage and step) and direct
  // loads L0 .. L1-1 of a refill (`is`), alternating and spread evenly over
  // all ops but the last two (so that the reads have returned by the end of
  // the step).  A wave issues in order, so a burst of reads or loads ahead
  // of the ops would leave the matrix cores idle while it is issued; spread
  // out, each instruction issues while an op is executing.  Scheduling
  // barriers keep this order (the compiler would otherwise sink the reads of
  // the next step below the ops of this one).
  struct FragSrc {
    int s, kk;
  };
  auto mfmas = [&](auto set, auto has_fr, auto lrange, const FragSrc& frs, const Issue& is) {
    constexpr int T = decltype(set)::value;
    using Other = std::integral_constant<int, 1 - T>;
    constexpr int L0 = decltype(lrange)::first, L1 = decltype(lrange)::second;
    constexpr int NF = decltype(has_fr)::value ? NFR : 0;
    constexpr int NL = L1 - L0;
    constexpr int M = NF + NL;
    constexpr int Q = F::FM * F::FN;
    constexpr int QS = Q > 4 ? Q - 2 : Q;  // ops followed by memory instructions
    constexpr int m = NF < NL ? NF : NL;   // pairs
    // CVTB: B fragment ni (read F(1 + ni)) is widened after op
    // min(qr + kCvtLag, Q - 1), qr being the op its read follows
    constexpr auto cvt_op = [](int ni) {
      const int idx = 1 + ni;
      const int j = idx < m ? 2 * idx : idx + m;  // its place in the sequence
      int qr = QS - 1;
      for (int q = 0; q < QS; ++q)
        if (q * M / QS <= j && j < (q + 1) * M / QS) qr = q;
      return qr + kCvtLag < Q - 1 ? qr + kCvtLag : Q - 1;
    };
    __builtin_amdgcn_sched_barrier(0);
    StaticFor<0, Q>::run([&](auto qq) {
      constexpr int q = decltype(qq)::value;
      constexpr int mi = q / F::FN, ni = q % F::FN;
      f.acc[mi][ni] = Op::mfma(fa[T][mi], fb[T][ni], f.acc[mi][ni]);
      // memory instructions j0 .. j1-1 of the alternating sequence F0, L0,
      // F1, L1, ... (the longer list continuing alone)
      constexpr int j0 = q < QS ? q * M / QS : M, j1 = q < QS ? (q + 1) * M / QS : M;
      StaticFor<j0, j1>::run([&](auto jj) {
        constexpr int j = decltype(jj)::value;
        constexpr bool frag = j < 2 * m ? (j % 2 == 0) : (NF > NL);
        constexpr int idx = j < 2 * m ? j / 2 : j - m;
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (frag)
          read_frag(Other(), std::integral_constant<int, idx>(), frs.s, frs.kk);
        else
          issue_part(is, L0 + idx);
        __builtin_amdgcn_sched_barrier(0);
      });
      if constexpr (CVTB && NF > 0) {
        StaticFor<0, F::FN>::run([&](auto nn) {
          if constexpr (cvt_op(decltype(nn)::value) == q) {
            __builtin_amdgcn_sched_barrier(0);
            cvt_frag(Other(), nn);
            __builtin_amdgcn_sched_barrier(0);
          }
        });
      }
    });
    __builtin_amdgcn_sched_barrier(0);
  };

  int64_t nk = 0;      // K tiles of the current job
  int64_t issued = 0;  // K tiles whose loads have been issued
  bool prefetched = false;  // the current job's first K tiles were issued by the previous one
  constexpr int KS = KB / 16;  // K=16 steps per tile (even)
  // A refill's LPS loads are spread over the KS steps of the tile that
  // issues them: step k issues loads k LPS / KS .. (k + 1) LPS / KS - 1, so
  // PRE of them precede the barrier of the tile's last step.
  constexpr int PRE = (KS - 1) * LPS / KS;
  // Makes K tile `next` visible to every wave: wait for this wave's loads of
  // it (the STAGES - 3 tiles issued after it, and the PRE loads of the
  // current refill, may stay in flight) and for its LDS reads, then a bare
  // barrier (__syncthreads() would also wait for the loads still in flight).
  // After the barrier every wave has read the last fragments of tile
  // next - 1, so the buffer of tile next - 1 is free: the refill with tile
  // next + STAGES - 1 that the next tile issues may start at once.
  static_assert(STAGES >= 3, "one buffer being read, one about to be read, one or more in flight");
  static_assert((STAGES - 3) * LPS + PRE < 64, "vmcnt holds at most 63 outstanding loads");
  auto sync_tile = [&](int64_t next, auto tail) {
    if constexpr (decltype(tail)::value) {
      const int64_t after = issued - 1 - next;  // 0 .. STAGES - 3
      StaticFor<0, STAGES - 2>::run([&](auto q) {
        constexpr int n = decltype(q)::value;
        if (after == n) wait_vmcnt_lds<n * LPS>();
      });
    } else {
      wait_vmcnt_lds<(STAGES - 3) * LPS + PRE>();
    }
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  using True = std::integral_constant<bool, true>;
  using False = std::integral_constant<bool, false>;
  using Set0 = std::integral_constant<int, 0>;
  // K tile i (fragments of its first step already requested into set 0).
  // has_next: tile i + 1 exists; refill: tile i + STAGES - 1 exists (into
  // the buffer of tile i - 1, free since the barrier before this tile).
  auto tile = [&](int64_t i, auto has_next, auto refill, auto tail) {
    const int s = static_cast<int>(i % STAGES);
    Issue is{};
    if constexpr (decltype(refill)::value) {
      is = issue_begin(static_cast<int>(issued % STAGES));
      ++issued;
    }
    StaticFor<0, KS>::run([&](auto kq) {
      constexpr int kk = decltype(kq)::value;
      using Cur = std::integral_constant<int, kk & 1>;
      constexpr int la = decltype(refill)::value ? kk * LPS / KS : 0;
      constexpr int lb = decltype(refill)::value ? (kk + 1) * LPS / KS : 0;
      if constexpr (kk + 1 < KS) {
        mfmas(Cur(), True(), LoadRange<la, lb>(), FragSrc{s, kk + 1}, is);
      } else if constexpr (decltype(has_next)::value) {
        sync_tile(i + 1, tail);
        mfmas(Cur(), True(), LoadRange<la, lb>(), FragSrc{static_cast<int>((i + 1) % STAGES), 0}, is);
      } else {
        mfmas(Cur(), False(), LoadRange<la, lb>(), FragSrc{0, 0}, is);
      }
    });
  };

  for (int job = 0; job < njobs; ++job) {
    if constexpr (PAIRED) {
      // job 0: K tiles from the last one down to the diagonal block of its
      // row tile.  job 1: K tiles from the block right of its diagonal block
      // up to the last one, then its diagonal block downwards.  At any time
      // the workgroups of one column tile then read at most two K blocks of
      // B (block T - 1 - s in job 0, block s in job 1, s counted in blocks
      // from the start), and every job ends on its diagonal block in
      // descending order (the epilogue finds the last K tiles of that block
      // still staged).
      const int64_t kpb = BM / KB;  // K tiles per K block
      if (job == 0) {
        nk = ktiles - f.tm * kpb;
        tw.init(p, f.z, f.tm, f.tn, BM, BN, ktiles - 1, false, -1, 0);
      } else {
        f.tm = tm1;
        f.tn = tn1;
        const int64_t lo = f.tm * kpb;
        const int64_t hi = lo + kpb < ktiles ? lo + kpb : ktiles;
        const int64_t up = ktiles - hi;
        nk = up + (hi - lo);
        if (up > 0)
          tw.init(p, f.z, f.tm, f.tn, BM, BN, hi, true, up, hi - 1);
        else
          tw.init(p, f.z, f.tm, f.tn, BM, BN, hi - 1, false, -1, 0);
      }
    } else {
      nk = kt1 - kt0;
    }
    f.row0 = f.tm * BM + f.wm * F::WM;
    f.col0 = f.tn * BN + f.wn * F::WN;
#pragma unroll
    for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
      for (int ni = 0; ni < F::FN; ++ni)
#pragma unroll
        for (int r = 0; r < 16; ++r) f.acc[mi][ni][r] = 0.0f;
    if (!PERSIST || !prefetched) {
      set_offsets(f.tm, f.tn);
      issued = 0;
      if (nk > 0) {
        if constexpr (!PAIRED) kp.init(p, kt0, f.z, f.tm, f.tn, BM, BN);
        // tiles 0 .. STAGES - 3 up front, tile STAGES - 2 once tile 0 is visible
        for (int q = 0; q < STAGES - 2 && issued < nk; ++q) {
          issue(q);
          ++issued;
        }
      }
    }
    if (nk > 0) {
      sync_tile(0, True());
      if (issued < nk) {
        issue(STAGES - 2);
        ++issued;
      }
      read_frags(Set0(), 0, 0);
      int64_t i = 0;
      for (; i + STAGES - 1 < nk; ++i) tile(i, True(), True(), False());
      for (; i + 1 < nk; ++i) tile(i, True(), False(), True());
      tile(i, False(), False(), True());
    }
    // Pin the accumulators to AGPRs across the loop: otherwise an epilogue
    // that feeds them to VALU instructions can pull part of them into VGPRs,
    // which the loop then runs out of.
#pragma unroll
    for (int mi = 0; mi < F::FM; ++mi)
#pragma unroll
      for (int ni = 0; ni < F::FN; ++ni) asm volatile("" : "+a"(f.acc[mi][ni]));
    // Persistent launch with an epilogue that leaves the LDS alone: once
    // every wave is done with the stage buffers, the first K tiles of the
    // next tile are issued into them, and the epilogue's stores go out
    // behind those loads.
    bool pre = false;
    int ntm = 0, ntn = 0, nks = 0;
    int64_t nz = 0;
    if constexpr (PERSIST) {
      if (job + 1 < njobs) {
        __syncthreads();  // every wave's fragment reads of this tile returned
        flat_coords(pjob0 + static_cast<int64_t>(job + 1) * pstride, &ntm, &ntn, &nz, &nks);
        const int64_t nkt0 = ktiles * nks / p.splits, nkt1 = ktiles * (nks + 1) / p.splits;
        set_offsets(ntm, ntn);
        issued = 0;
        if (nkt1 > nkt0) {
          kp.init(p, nkt0, nz, ntm, ntn, BM, BN);
          for (int q = 0; q < STAGES - 2 && issued < nkt1 - nkt0; ++q) {
            issue(q);
            ++issued;
          }
        }
        pre = true;
      }
    }
    if (!pre) {
      wait_vmcnt<0>();
      __syncthreads();  // epilogues may reuse the stage buffers
    }
    StageLds lds;
    lds.a = As;
    lds.b = Bs;
    lds.a_elems = STAGES * ASZ;
    lds.b_elems = STAGES * BSZ;
    lds.nk = nk;
    lds.stages = STAGES;
    epi(f, lds);
    if constexpr (PAIRED) __syncthreads();  // the next job refills the stage buffers
    if constexpr (PERSIST) {
      if (pre) {
        f.tm = ntm;
        f.tn = ntn;
        f.z = nz;
        f.ks = nks;
        kt0 = ktiles * nks / p.splits;
        kt1 = ktiles * (nks + 1) / p.splits;
      }
      prefetched = pre;
    }
  }
}

}  // namespace gemm
}  // namespace bitsmoe
