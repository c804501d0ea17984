// Linear layer with a fused ReGELU2 / ReSiLU2 forward epilogue, for gfx950.
//
// z = x W^T (+ b): x [M x K] and W [N x K] (the weight of a linear layer) are bf16
// and K-contiguous; products accumulate in fp32 on v_mfma_f32_32x32x16_bf16 and z is
// rounded once to bf16 (bias added in fp32 before the rounding). The epilogue then
// applies the activation to the rounded z and stores y = act(z) and the 2-bit codes
// of z (Sec. 4.2; 16 codes per word over the flattened [M x N] output), i.e. exactly
// what the activation kernels compute from a stored z. z itself is stored only when
// the caller asks for it: ReGELU2 / ReSiLU2 keep only the codes for the backward
// pass, so the pre-activation never has to reach HBM.
//
// Tiling. A block computes a BM x BN tile of z with WM x WN waves, each a
// (BM/WM) x (BN/WN) part as 32 x 32 MFMA tiles, accumulators in registers. Two tile
// configurations are compiled and chosen per problem (launcher): 256 x 256 with 8 waves
// of 128 x 64 for large problems, 128 x 128 with 8 waves of 64 x 32 (two blocks per CU)
// when the large tiles would leave much of the last round of the GPU idle.
//
// K loop. K advances in steps of BK = 64 (32 also compiles) through a ring of LDS stages
// (two for the shipped configurations) filled straight from HBM by raw buffer loads
// with an LDS destination (buffer_load_dwordx4 ... lds), so no register staging is
// needed; the longer step halves the block barriers per flop, which is what the matrix
// cores were waiting on. The buffer resources end at the tile's last valid row, so
// ragged tiles read zeros without branches, and chunks beyond K are pointed past the end
// to read zeros too. A stage row is BK bf16 = U = BK / 8 sixteen-byte units, unit u of
// row r holding k-chunk u ^ ((r >> s) % U), with 2^s rows per 256 bytes, so that the
// operand reads of 16 consecutive rows at one k-chunk hit distinct LDS banks; one load
// instruction of a wave fills 1 KiB (64 / U rows), lane l writing unit l % U of row
// l / U (the row's U lanes read its 2 BK contiguous bytes in permuted order). Within the loop the fragments of the next K slice (16) are read into
// their own registers while the MFMAs of the current one run (scheduling groups put one
// MFMA between consecutive loads and reads), across step boundaries too; the loop body
// is branch-free (loads past the last step read zeros into spent
// buffers) so that the compiler's LDS waits are exact. Lane layout of the MFMA (checked
// on the hardware): lane l supplies row l % 32 of A and column l % 32 of B at
// k = 8 (l / 32) .. + 7, and holds result rows 8 (r / 4) + 4 (l / 32) + r % 4 of column
// l % 32 in accumulator register r.
//
// Epilogue: the tile (bias added, rounded to bf16) is written to LDS and read back so
// that each thread owns 16 consecutive columns of a row: two 16-byte stores of y (and
// of z), one code word, the same arithmetic as the activation kernels' fast path.
//
// Blocks are mapped to tiles XCD by XCD (the hardware deals consecutive blocks out
// to the 8 XCDs in turn), in groups of 8 row tiles, so that the blocks sharing an XCD's
// L2 also share their x and W tiles.
#include "lmbp_device.hpp"
#include "act_codes.hpp"
#include "act_math.hpp"
#include "lmbp_launch.hpp"

#include <atomic>

namespace lmbp {
namespace lin {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kXcds = 8;
constexpr int kGroupM = 8;
constexpr uint32_t kBufferGDword3 = 0x00020000;  // raw 32-bit buffer, gfx9 family
constexpr uint32_t kOutOfRange = 0x80000000u;    // beyond any resource's range: reads 0

template <int BM_, int BN_, int WM_, int WN_, int STAGES_ = 4, int BK_ = 32>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int kStages = STAGES_;   // LDS ring
  static constexpr int BK = BK_;            // K step: a stage row is 2 BK bytes
  static constexpr int kSlices = BK / 16;   // MFMA K slices per step
  static constexpr int kUnits = BK / 8;     // 16-byte units per stage row
  static constexpr int kRowsPerLoad = 64 / kUnits;            // rows one 1 KiB load fills
  static constexpr int kSwzShift = BK == 32 ? 2 : 1;          // rows per 256 bytes: 4 or 2
  static_assert(BK == 32 || BK == 64, "K step of 32 or 64");
  static constexpr int kWaves = WM * WN;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int TM = BM / WM / 32, TN = BN / WN / 32;   // MFMA tiles per wave
  static constexpr int kStageElems = (BM + BN) * BK;
  static constexpr int kEpiRow = BN + 8;                        // padded epilogue row
  static constexpr int kOperandElems = kStages * kStageElems;
  static constexpr int kLdsElems =
      (kOperandElems > BM * kEpiRow) ? kOperandElems : BM * kEpiRow;
  static constexpr int kLdsElemsNorm = kLdsElems + 2 * BM;   // + the rows' rstd (fp32)
  static constexpr int kLA = BM / kRowsPerLoad / kWaves, kLB = BN / kRowsPerLoad / kWaves;
  static constexpr int kLoadsPerStage = kLA + kLB;
  static constexpr int kEpiThreadsPerRow = BN / 16;
  static constexpr int kEpiRowStep = kThreads / kEpiThreadsPerRow;
  static_assert(BM % (WM * 32) == 0 && BN % (WN * 32) == 0, "wave tiles are multiples of 32");
  static_assert((BM / kRowsPerLoad) % kWaves == 0 && (BN / kRowsPerLoad) % kWaves == 0,
                "load blocks per wave");
  static_assert(kThreads % kEpiThreadsPerRow == 0, "epilogue mapping");
  static_assert(kLdsElemsNorm * 2 <= 160 * 1024, "LDS per block");
  static_assert(kStages >= 2 && (kStages - 1) * kLoadsPerStage <= 63, "vector-memory counter range");
};

#ifndef LMBP_LIN_SMALL
#define LMBP_LIN_SMALL 128, 128, 2, 4, 2, 64   // the same for the small configuration (8 waves)
#endif
#ifndef LMBP_LIN_BIG
#define LMBP_LIN_BIG 256, 256, 2, 4, 2, 64   // BM, BN, WM, WN, stages, K step: large configuration
#endif
using BigTile = Tile<LMBP_LIN_BIG>;
using SmallTile = Tile<LMBP_LIN_SMALL>;

// The target builtins below are wrapped in device functions: used directly in the body of
// a kernel template, they make the host-side instantiation fail silently and the launch
// stub is never emitted.

// A raw buffer resource over `bytes` bytes at `base` (reads beyond return zeros).
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const uint16_t* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, int(bytes),
                                           kBufferGDword3);
}

// 16 bytes per lane from the buffer into LDS at `dst` + lane * 16 (dst wave-uniform).
__device__ inline void load_lds16(__amdgpu_buffer_rsrc_t r, uint16_t* dst, uint32_t offset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, offset, 0, 0, 0);
}

// Scheduling groups for one K slice: its MF MFMAs, with VM buffer loads and then DS LDS
// reads spread over the first half of them (so the reads have landed before the slice
// ends and the next wait finds nothing outstanding).
template <int MF, int VM, int DS, int I = 0>
__device__ inline void spread() {
  if constexpr (I < MF) {
    constexpr int W = MF / 2 < 1 ? 1 : MF / 2;
    constexpr int T = VM + DS;
    constexpr int lo = I < W ? T * I / W : T, hi = I < W ? T * (I + 1) / W : T;
    constexpr int vm = (hi < VM ? hi : VM) - (lo < VM ? lo : VM);
    constexpr int ds = (hi - lo) - vm;
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                  // one MFMA
    if constexpr (vm > 0) __builtin_amdgcn_sched_group_barrier(0x020, vm, 0);  // buffer loads
    if constexpr (ds > 0) __builtin_amdgcn_sched_group_barrier(0x100, ds, 0);  // LDS reads
    spread<MF, VM, DS, I + 1>();
  }
}

// Tile coordinates of this block (see the file comment).
__device__ inline void block_tile(int64_t tiles_m, int64_t tiles_n, int64_t& tm, int64_t& tn) {
  const int64_t nblk = tiles_m * tiles_n;
  const int64_t b = blockIdx.x;
  const int64_t per = nblk / kXcds;
  const int64_t id = (b < per * kXcds) ? (b % kXcds) * per + b / kXcds : b;
  const int64_t in_group = kGroupM * tiles_n;
  const int64_t first_m = (id / in_group) * kGroupM;
  const int64_t gsize = (tiles_m - first_m < kGroupM) ? tiles_m - first_m : kGroupM;
  const int64_t r = id % in_group;
  tm = first_m + r % gsize;
  tn = r / gsize;
}

// Arguments of the kernel (by value). Plain form: y = act(z), z = x w^T + bias.
// Gated form (GLU): g = x w^T and u = x w2^T (no bias), y = h = act(g) * u, s = act(g),
// u stored; z (optional) receives g; codes are those of g.
struct LinArgs {
  const uint16_t* x;
  const uint16_t* w;
  const uint16_t* w2;
  const uint16_t* bias;
  uint16_t* y;
  uint16_t* s;
  uint16_t* u;
  uint32_t* codes;
  uint16_t* z;
  int64_t M, N, K;
  // Norm in front (NORM): x is the norm's input, rstd its per-row statistic (fp32), and
  // zn [M x K] receives the norm's output z = bf16(x rstd).
  const float* rstd;
  uint16_t* zn;
};

template <class C, int ACT, bool GLU, bool NORM>
__global__ __launch_bounds__(C::kThreads) void linear_act_fwd_kernel(LinArgs a) {
  using A = ActOf<ACT>;
  constexpr int BM = C::BM, BN = C::BN, TM = C::TM, TN = C::TN, kWaves = C::kWaves;
  // Output columns per block: the gated form spends half of the B tile on each weight.
  constexpr int kOut = GLU ? BN / 2 : BN;
  static_assert(!GLU || C::kLB % 2 == 0, "gated form: each weight fills half the B loads");
  const uint16_t* __restrict__ x = a.x;
  const uint16_t* __restrict__ w = a.w;
  const int64_t M = a.M, N = a.N, K = a.K;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int wm = wave / C::WN, wn = wave % C::WN;

  int64_t tm, tn;
  const int64_t tiles_n = (N + kOut - 1) / kOut;
  block_tile((M + BM - 1) / BM, tiles_n, tm, tn);
  const int64_t m0 = tm * BM, n0 = tn * kOut;

  // Norm in front: the block's rows' rstd in LDS past the operand / epilogue area
  // (visible after the first barrier).
  float* rs_lds = reinterpret_cast<float*>(lds + C::kLdsElems);
  if constexpr (NORM) {
    for (int r = tid; r < BM; r += C::kThreads) rs_lds[r] = (m0 + r < M) ? a.rstd[m0 + r] : 0.0f;
  }

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Buffer resources over the block's rows of x and W.
  const int64_t rows_x = (M - m0 < BM) ? M - m0 : BM;
  const int64_t rows_w = (N - n0 < kOut) ? N - n0 : kOut;
  const auto rx = make_rsrc(x + m0 * K, rows_x * K * 2);
  const auto rw = make_rsrc(w + n0 * K, rows_w * K * 2);
  const auto rw2 = make_rsrc(GLU ? a.w2 + n0 * K : w, GLU ? rows_w * K * 2 : 0);

  // Loads: lane l of the wave's q-th 1 KiB block (stage rows R (wave + waves q) + l / U,
  // R rows of U units) fetches k-chunk kc = (l % U) ^ swz(row) of its row, so that unit u
  // of stage row r holds chunk u ^ swz(r), swz(r) = (r >> kSwzShift) % U.
  const int r_in = lane / C::kUnits;
  const int u_in = lane % C::kUnits;
  auto chunk = [&](int stage_row) { return u_in ^ ((stage_row >> C::kSwzShift) & (C::kUnits - 1)); };
  uint32_t ld_a[C::kLA], ld_b[C::kLB];  // byte offset of the chunk at K step 0
  int kc_a[C::kLA], kc_b[C::kLB];
#pragma unroll
  for (int q = 0; q < C::kLA; ++q) {
    const int row = (wave + kWaves * q) * C::kRowsPerLoad + r_in;
    kc_a[q] = chunk(row);
    ld_a[q] = uint32_t(row * K * 2 + kc_a[q] * 16);
  }
  // Gated form: B-tile rows below BN / 2 come from w, the others (the second half of the
  // loads, q >= kLB / 2) from w2, each at its own row offset.
#pragma unroll
  for (int q = 0; q < C::kLB; ++q) {
    const int srow = (wave + kWaves * q) * C::kRowsPerLoad + r_in;
    kc_b[q] = chunk(srow);
    const int row = srow - ((GLU && q >= C::kLB / 2) ? BN / 2 : 0);
    ld_b[q] = uint32_t(row * K * 2 + kc_b[q] * 16);
  }
  constexpr int kStages = C::kStages;
  auto stage_ptr = [&](int64_t kt) { return lds + int(kt % kStages) * C::kStageElems; };
  auto issue_stage = [&](int64_t kt) {
    uint16_t* S = stage_ptr(kt);
    const uint32_t k0b = uint32_t(kt * C::BK * 2);
#pragma unroll
    for (int q = 0; q < C::kLA; ++q)
      load_lds16(rx, S + (wave + kWaves * q) * 512,
                 kt * C::BK + kc_a[q] * 8 < K ? ld_a[q] + k0b : kOutOfRange);
#pragma unroll
    for (int q = 0; q < C::kLB; ++q)
      load_lds16((GLU && q >= C::kLB / 2) ? rw2 : rw, S + BM * C::BK + (wave + kWaves * q) * 512,
                 kt * C::BK + kc_b[q] * 8 < K ? ld_b[q] + k0b : kOutOfRange);
  };

  // Operand reads: lane l reads row (base + l % 32), k-chunk 2 kk + l / 32; wave rows
  // start at multiples of 32, so the row's swizzle is ((l % 32) >> 2) & 3.
  const int swz = ((lane & 31) >> C::kSwzShift) & (C::kUnits - 1);
  int a_row[TM], b_row[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) a_row[i] = (wm * TM * 32 + i * 32 + (lane & 31)) * C::BK;
#pragma unroll
  for (int j = 0; j < TN; ++j) b_row[j] = BM * C::BK + (wn * TN * 32 + j * 32 + (lane & 31)) * C::BK;
  bf16x8 fa[2][TM], fb[2][TN];
  auto read = [&](const uint16_t* S, int kk, int buf) {
    const int unit = ((2 * kk + (lane >> 5)) ^ swz) * 8;
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[buf][i] = *reinterpret_cast<const bf16x8*>(S + a_row[i] + unit);
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[buf][j] = *reinterpret_cast<const bf16x8*>(S + b_row[j] + unit);
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[buf][i], fb[buf][j], acc[i][j], 0, 0, 0);
  };

  // Norm in front: the norm's output z = bf16(x rstd), stored with the norm kernel's
  // rounding (fp32 product, round to nearest even). The x columns of K step kt of this
  // row tile are written by the block with tn = kt mod tiles_n, from x read again (it
  // has just streamed through the caches), outside the K loop, whose body stays
  // branch-free. The block's first chunk is requested before the last K step's matrix
  // products, which hide the loads. Consecutive lanes take consecutive 16-byte chunks of
  // a row; rows beyond M and columns beyond K read through an empty range (zeros).
  constexpr int kZv = NORM ? BM * (C::BK / 8) / C::kThreads : 1;
  u32x4 zv[kZv];
  auto z_chunk_load = [&](int64_t kt) {
    constexpr int U = C::BK / 8;
    const auto r = make_rsrc(x + m0 * K, rows_x * K * 2);
#pragma unroll
    for (int i = 0; i < kZv; ++i) {
      const int q = tid + i * C::kThreads;
      const int64_t col = kt * C::BK + (q % U) * 8;
      zv[i] = __builtin_amdgcn_raw_buffer_load_b128(
          r, col < K ? uint32_t(((q / U) * K + col) * 2) : kOutOfRange, 0, 0);
    }
  };
  auto z_chunk_store = [&](int64_t kt) {
    constexpr int U = C::BK / 8;
#pragma unroll
    for (int i = 0; i < kZv; ++i) {
      const int q = tid + i * C::kThreads;
      const int rr = q / U;
      const int64_t col = kt * C::BK + (q % U) * 8;
      if (m0 + rr < M && col < K) {
        const float rsr = rs_lds[rr];
        float f[8];
        BF16::unpack(zv[i], f);
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = f[e] * rsr;
        *reinterpret_cast<u32x4*>(a.zn + (m0 + rr) * K + col) = BF16::pack(f);
      }
    }
  };

  // Loads of steps at or beyond the last one read zeros into buffers that are no longer
  // needed, so every step sees the same number of loads in flight and the waits are
  // constants (the vector-memory counter counts only these loads in the loop).
  constexpr int kPendingFirst = (kStages - 1) * C::kLoadsPerStage;    // loads after step 0
  constexpr int kPendingSteady = (kStages - 2) * C::kLoadsPerStage;   // after step kt + 1
  const int64_t kt_count = (K + C::BK - 1) / C::BK;
  if (kt_count > 0) {
#pragma unroll
    for (int s = 0; s < kStages; ++s) issue_stage(s);
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(kPendingFirst) : "memory");
    asm volatile("s_barrier" ::: "memory");
    read(stage_ptr(0), 0, 0);
    for (int64_t kt = 0; kt + 1 < kt_count; ++kt) {
      const uint16_t* S = stage_ptr(kt);
#pragma unroll
      for (int kk = 0; kk < C::kSlices; ++kk) {
        if (kk + 1 < C::kSlices) {
          read(S, kk + 1, (kk + 1) & 1);
          mfmas(kk & 1);
          spread<TM * TN, 0, TM + TN>();
        } else {
          // This wave's reads of step kt are complete once their data has arrived; after
          // the barrier every wave's are, and step kt + 1 is in LDS.
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          asm volatile("s_waitcnt vmcnt(%0)" :: "n"(kPendingSteady) : "memory");
          asm volatile("s_barrier" ::: "memory");
          issue_stage(kt + kStages);   // into step kt's buffer
          read(stage_ptr(kt + 1), 0, 0);
          mfmas(kk & 1);
          spread<TM * TN, C::kLoadsPerStage, TM + TN>();
        }
        __builtin_amdgcn_sched_barrier(0);   // the slice's MFMAs stay ahead of the next wait
      }
    }
    const uint16_t* S = stage_ptr(kt_count - 1);
    if constexpr (NORM) {
      if (tn < kt_count) z_chunk_load(tn);
    }
#pragma unroll
    for (int kk = 0; kk < C::kSlices; ++kk) {
      if (kk + 1 < C::kSlices) read(S, kk + 1, (kk + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
      mfmas(kk & 1);
    }
  }
  __syncthreads();   // waits for every load (including the zero-filling ones) and read

  if constexpr (NORM) {
    for (int64_t kt = tn; kt < kt_count; kt += tiles_n) {
      if (kt != tn) z_chunk_load(kt);
      z_chunk_store(kt);
    }
  }

  // Epilogue, part 1: bias, rounding to bf16, the tile into LDS (row-major, padded).
  // Gated form: columns [0, BN/2) hold g, [BN/2, BN) hold u of the same output columns.
  uint16_t* E = lds;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int col = wn * TN * 32 + j * 32 + (lane & 31);
    const float bj = (!GLU && a.bias != nullptr && n0 + col < N)
                         ? __uint_as_float(uint32_t(a.bias[n0 + col]) << 16) : 0.0f;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * TM * 32 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        // norm in front: z W^T = rstd (x W^T), the row scale applied to the fp32 sum
        const float v = NORM ? __builtin_fmaf(acc[i][j][r], rs_lds[row], bj) : acc[i][j][r] + bj;
        E[row * C::kEpiRow + col] = uint16_t(pack_bf16x2(v, 0.0f) & 0xffffu);
      }
  }
  __syncthreads();

  // Part 2: thread owns output columns c16 .. c16 + 15 of rows tid / (kOut/16) + step * g.
  constexpr int kTpr = kOut / 16;
  static_assert(C::kThreads % kTpr == 0, "epilogue mapping");
  const int c16 = (tid % kTpr) * 16;
  if (n0 + c16 >= N) return;  // N is a multiple of 16: a group is wholly in or out
  for (int row = tid / kTpr; row < BM; row += C::kThreads / kTpr) {
    if (m0 + row >= M) break;
    const u32x4 v0 = *reinterpret_cast<const u32x4*>(E + row * C::kEpiRow + c16);
    const u32x4 v1 = *reinterpret_cast<const u32x4*>(E + row * C::kEpiRow + c16 + 8);
    float f0[8], f1[8], o0[8], o1[8];
    BF16::unpack(v0, f0);
    BF16::unpack(v1, f1);
    const int64_t base = (m0 + row) * N + n0 + c16;   // flat element index, multiple of 16
    if constexpr (GLU) {
      // Same arithmetic as the SwiGLU activation kernel on stored g and u.
      const u32x4 u0 = *reinterpret_cast<const u32x4*>(E + row * C::kEpiRow + BN / 2 + c16);
      const u32x4 u1 = *reinterpret_cast<const u32x4*>(E + row * C::kEpiRow + BN / 2 + c16 + 8);
      float g0[8], g1[8];
      BF16::unpack(u0, g0);
      BF16::unpack(u1, g1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        gated_value<ACT, false>(f0[e], g0[e], o0[e], g0[e]);
        gated_value<ACT, false>(f1[e], g1[e], o1[e], g1[e]);
      }
      *reinterpret_cast<u32x4*>(a.y + base) = BF16::pack(g0);
      *reinterpret_cast<u32x4*>(a.y + base + 8) = BF16::pack(g1);
      *reinterpret_cast<u32x4*>(a.s + base) = BF16::pack(o0);
      *reinterpret_cast<u32x4*>(a.s + base + 8) = BF16::pack(o1);
      *reinterpret_cast<u32x4*>(a.u + base) = u0;
      *reinterpret_cast<u32x4*>(a.u + base + 8) = u1;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        o0[e] = act_value<ACT, false>(f0[e]);
        o1[e] = act_value<ACT, false>(f1[e]);
      }
      *reinterpret_cast<u32x4*>(a.y + base) = BF16::pack(o0);
      *reinterpret_cast<u32x4*>(a.y + base + 8) = BF16::pack(o1);
    }
    a.codes[base / 16] = codes_of<A>(f0) | (codes_of<A>(f1) << 16);
    if (a.z != nullptr) {
      *reinterpret_cast<u32x4*>(a.z + base) = v0;
      *reinterpret_cast<u32x4*>(a.z + base + 8) = v1;
    }
  }
}

template <class C, int ACT, bool GLU, bool NORM = false>
hipError_t launch_tile(const LinArgs& a, hipStream_t s) {
  constexpr int kOut = GLU ? C::BN / 2 : C::BN;
  const int64_t blocks = ((a.M + C::BM - 1) / C::BM) * ((a.N + kOut - 1) / kOut);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  const size_t lds = size_t(NORM ? C::kLdsElemsNorm : C::kLdsElems) * 2;
  // More than 64 KiB of dynamic LDS must be allowed explicitly, per kernel and device;
  // the attribute is set on the first launch on each device.
  constexpr int kMaxDevices = 64;
  static std::atomic<bool> attr_set[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (!attr_set[dev].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(linear_act_fwd_kernel<C, ACT, GLU, NORM>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    attr_set[dev].store(true, std::memory_order_release);
  }
  hipLaunchKernelGGL((linear_act_fwd_kernel<C, ACT, GLU, NORM>), dim3(unsigned(blocks)),
                     dim3(C::kThreads), lds, s, a);
  return hipGetLastError();
}

#ifndef LMBP_LIN_BIG_MIN_ROUNDS
// Use the 256 x 256 tiles when they fill at least this many rounds of the GPU's CUs
// (one block per CU); otherwise the 128 x 128 tiles (two blocks per CU) waste less of the
// last round. Measured: the ViT-B MLP projection (2.3 rounds) runs faster with the small
// tiles, the LLaMA-7B gate projection (5.4 rounds) with the large ones.
#define LMBP_LIN_BIG_MIN_ROUNDS 4
#endif

}  // namespace lin

namespace {
// Large tiles when they fill at least LMBP_LIN_BIG_MIN_ROUNDS rounds of the CUs.
bool use_big_tiles(int64_t M, int64_t N_tile_cols) {
  int device = 0, cus = 256;
  if (hipGetDevice(&device) == hipSuccess)
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
  const int64_t big_tiles = ((M + lin::BigTile::BM - 1) / lin::BigTile::BM) *
                            ((N_tile_cols + lin::BigTile::BN - 1) / lin::BigTile::BN);
  return big_tiles >= int64_t(LMBP_LIN_BIG_MIN_ROUNDS) * cus;
}
}  // namespace

hipError_t launch_linear_act_fwd(int act, int64_t M, int64_t N, int64_t K, const void* x,
                                 const void* w, const void* bias, void* y, uint32_t* codes,
                                 void* z, hipStream_t s) {
  lin::LinArgs a{static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w), nullptr,
                 static_cast<const uint16_t*>(bias), static_cast<uint16_t*>(y), nullptr,
                 nullptr, codes, static_cast<uint16_t*>(z), M, N, K, nullptr, nullptr};
  const bool big = use_big_tiles(M, N);
  using lin::BigTile;
  using lin::SmallTile;
  using lin::launch_tile;
  if (act == kGelu)
    return big ? launch_tile<BigTile, kGelu, false>(a, s) : launch_tile<SmallTile, kGelu, false>(a, s);
  return big ? launch_tile<BigTile, kSilu, false>(a, s) : launch_tile<SmallTile, kSilu, false>(a, s);
}

hipError_t launch_linear_glu_fwd(int64_t M, int64_t N, int64_t K, const void* x, const void* w_gate,
                                 const void* w_up, void* h, void* s_out, void* u, uint32_t* codes,
                                 void* g, hipStream_t s) {
  lin::LinArgs a{static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w_gate),
                 static_cast<const uint16_t*>(w_up), nullptr, static_cast<uint16_t*>(h),
                 static_cast<uint16_t*>(s_out), static_cast<uint16_t*>(u), codes,
                 static_cast<uint16_t*>(g), M, N, K, nullptr, nullptr};
  // Each block covers half as many output columns as its tile width.
  const bool big = use_big_tiles(M, 2 * N);
  return big ? lin::launch_tile<lin::BigTile, kSilu, true>(a, s)
             : lin::launch_tile<lin::SmallTile, kSilu, true>(a, s);
}

hipError_t launch_linear_rms_act_fwd(int act, int64_t M, int64_t N, int64_t K, float eps,
                                     const void* x, const void* w, const void* bias, void* y,
                                     uint32_t* codes, void* pre, void* z_norm, float* rstd,
                                     hipStream_t s) {
  hipError_t e = launch_norm_fwd(false, true, M, K, eps, x, nullptr, rstd, true, s);
  if (e != hipSuccess) return e;
  lin::LinArgs a{static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w), nullptr,
                 static_cast<const uint16_t*>(bias), static_cast<uint16_t*>(y), nullptr,
                 nullptr, codes, static_cast<uint16_t*>(pre), M, N, K, rstd,
                 static_cast<uint16_t*>(z_norm)};
  const bool big = use_big_tiles(M, N);
  using lin::BigTile;
  using lin::SmallTile;
  using lin::launch_tile;
  if (act == kGelu)
    return big ? launch_tile<BigTile, kGelu, false, true>(a, s) : launch_tile<SmallTile, kGelu, false, true>(a, s);
  return big ? launch_tile<BigTile, kSilu, false, true>(a, s) : launch_tile<SmallTile, kSilu, false, true>(a, s);
}

hipError_t launch_linear_rms_glu_fwd(int64_t M, int64_t N, int64_t K, float eps, const void* x,
                                     const void* w_gate, const void* w_up, void* h, void* s_out,
                                     void* u, uint32_t* codes, void* g, void* z_norm, float* rstd,
                                     hipStream_t s) {
  hipError_t e = launch_norm_fwd(false, true, M, K, eps, x, nullptr, rstd, true, s);
  if (e != hipSuccess) return e;
  lin::LinArgs a{static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w_gate),
                 static_cast<const uint16_t*>(w_up), nullptr, static_cast<uint16_t*>(h),
                 static_cast<uint16_t*>(s_out), static_cast<uint16_t*>(u), codes,
                 static_cast<uint16_t*>(g), M, N, K, rstd, static_cast<uint16_t*>(z_norm)};
  const bool big = use_big_tiles(M, 2 * N);
  return big ? lin::launch_tile<lin::BigTile, kSilu, true, true>(a, s)
             : lin::launch_tile<lin::SmallTile, kSilu, true, true>(a, s);
}

}  // namespace lmbp
