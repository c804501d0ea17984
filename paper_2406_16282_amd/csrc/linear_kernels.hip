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
// Tiling (defaults; measured best of the shapes tried on the LLaMA-7B gate and ViT-B
// MLP projections): a 512-thread block computes a 256 x 256 tile of z, its eight waves
// (4 along the rows, 2 along the columns) a 64 x 128 part each as 2 x 4 MFMA tiles of
// 32 x 32, accumulators in registers. K advances in steps of 32 through a ring of four
// LDS stages filled straight from HBM by raw buffer loads with an LDS destination
// (buffer_load_dwordx4 ... lds): three steps of loads are in flight ahead of the MFMAs
// and no register staging is needed. The buffer resources end at the tile's last valid
// row, so ragged tiles read zeros without branches. Each stage row is 64 bytes with an
// XOR swizzle of its four 16-byte units so that the operand reads of 16 consecutive
// rows hit distinct LDS banks. (A register-staged variant with padded rows and a
// two-step prefetch, LMBP_LIN_DIRECT=0, measured ~10% slower.) Lane layout of the MFMA
// (checked on the hardware): lane l supplies row l % 32 of A and column l % 32 of B at
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

namespace lmbp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#ifndef LMBP_LIN_BM
#define LMBP_LIN_BM 256  // block tile rows
#endif
#ifndef LMBP_LIN_BN
#define LMBP_LIN_BN 256  // block tile columns
#endif
#ifndef LMBP_LIN_WM
#define LMBP_LIN_WM 4    // waves along the rows of the tile
#endif
#ifndef LMBP_LIN_WN
#define LMBP_LIN_WN 2    // waves along the columns
#endif

#ifndef LMBP_LIN_PREFETCH
#define LMBP_LIN_PREFETCH 2  // K steps of global loads in flight ahead of the MFMAs (1 or 2)
#endif
#ifndef LMBP_LIN_DIRECT
#define LMBP_LIN_DIRECT 1  // 1: operands go from HBM straight to LDS (buffer_load ... lds)
#endif
#ifndef LMBP_LIN_STAGES
#define LMBP_LIN_STAGES 4  // LDS stages of the direct path
#endif
#ifndef LMBP_LIN_BK
#if LMBP_LIN_DIRECT
#define LMBP_LIN_BK 32   // the direct path's swizzle is laid out for 64-byte rows
#else
#define LMBP_LIN_BK 64   // K step (a multiple of 16)
#endif
#endif

constexpr int kBM = LMBP_LIN_BM, kBN = LMBP_LIN_BN, kBK = LMBP_LIN_BK;
constexpr int kWM = LMBP_LIN_WM, kWN = LMBP_LIN_WN;
constexpr int kThreads = kWM * kWN * kWave;
constexpr int kTM = kBM / kWM / 32;               // 32 x 32 MFMA tiles per wave, rows
constexpr int kTN = kBN / kWN / 32;               // and columns
constexpr int kLdsRow = kBK + 8;                  // bf16 per operand row in LDS (padded by 16 bytes)
constexpr int kKChunks = kBK / 8;                 // 16-byte chunks per row and K step
constexpr int kAElems = kBM * kLdsRow;            // one A buffer
constexpr int kBElems = kBN * kLdsRow;            // one B buffer
constexpr int kStageElems = kAElems + kBElems;
constexpr int kEpiRow = kBN + 8;                  // bf16 per row of the epilogue tile
#if LMBP_LIN_DIRECT
// Direct path: unpadded 64-byte rows (BK = 32) with an XOR swizzle of the 16-byte units.
static_assert(kBK == 32, "the direct path is laid out for K steps of 32");
constexpr int kStages = LMBP_LIN_STAGES;
constexpr int kDStageElems = (kBM + kBN) * kBK;
constexpr int kOperandElems = kStages * kDStageElems;
#else
// Two operand stages during the K loop.
constexpr int kOperandElems = 2 * kStageElems;
#endif
// The epilogue tile reuses the operand memory.
constexpr int kLdsElems = (kOperandElems > kBM * kEpiRow) ? kOperandElems : kBM * kEpiRow;
static_assert(kBM % (kWM * 32) == 0 && kBN % (kWN * 32) == 0, "wave tiles are multiples of 32");
constexpr int kChunksA = kBM * kBK / 8, kChunksB = kBN * kBK / 8;   // 16-byte chunks per step
static_assert(kChunksA % kThreads == 0 && kChunksB % kThreads == 0, "chunks per thread");
constexpr int kQA = kChunksA / kThreads, kQB = kChunksB / kThreads;
constexpr int kRowStep = kThreads / kKChunks;     // rows covered by one pass of the threads
static_assert((kThreads * 16) % kBN == 0, "epilogue mapping");
constexpr int kEpiThreadsPerRow = kBN / 16;
constexpr int kEpiRowStep = kThreads / kEpiThreadsPerRow;
constexpr int kXcds = 8;
constexpr int kGroupM = 8;

// One K step of both operands, 16-byte chunks: chunk c = tid + threads * q is row
// c / (BK/8), k-chunk c % (BK/8) of the tile. Loads are raw buffer loads against a resource
// that starts at the block's first row and ends after its last valid row, so rows
// beyond the matrix read zeros with no branch; chunks beyond K (K is a multiple of 8,
// so a chunk is wholly inside or outside) are pointed past the end to read zeros too.
struct Stage {
  u32x4 a[kQA], b[kQB];
};

struct Operands {
  __amdgpu_buffer_rsrc_t x, w;
  uint32_t xrow[kQA], wrow[kQB];  // byte offset of each chunk's row start
};

constexpr uint32_t kBufferGDword3 = 0x00020000;  // raw 32-bit buffer, gfx9 family
constexpr uint32_t kOutOfRange = 0x80000000u;

__device__ inline Operands make_operands(const uint16_t* x, const uint16_t* w, int64_t m0,
                                         int64_t n0, int64_t M, int64_t N, int64_t K) {
  Operands op;
  const int64_t rows_x = (M - m0 < kBM) ? M - m0 : kBM;
  const int64_t rows_w = (N - n0 < kBN) ? N - n0 : kBN;
  op.x = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(x) + m0 * K, 0,
                                           int(rows_x * K * 2), kBufferGDword3);
  op.w = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(w) + n0 * K, 0,
                                           int(rows_w * K * 2), kBufferGDword3);
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < kQA; ++q) op.xrow[q] = uint32_t((tid / kKChunks + kRowStep * q) * K * 2);
#pragma unroll
  for (int q = 0; q < kQB; ++q) op.wrow[q] = uint32_t((tid / kKChunks + kRowStep * q) * K * 2);
  return op;
}

__device__ inline void load_stage(Stage& st, const Operands& op, int64_t K, int64_t k0) {
  const int64_t k = k0 + (threadIdx.x % kKChunks) * 8;
  const uint32_t kb = uint32_t(k * 2);
  const bool kin = k < K;
#pragma unroll
  for (int q = 0; q < kQA; ++q)
    st.a[q] = __builtin_amdgcn_raw_buffer_load_b128(op.x, kin ? op.xrow[q] + kb : kOutOfRange, 0, 0);
#pragma unroll
  for (int q = 0; q < kQB; ++q)
    st.b[q] = __builtin_amdgcn_raw_buffer_load_b128(op.w, kin ? op.wrow[q] + kb : kOutOfRange, 0, 0);
}

__device__ inline void store_stage(const Stage& st, uint16_t* As, uint16_t* Bs) {
  const int tid = threadIdx.x;
  const int kc = tid % kKChunks;
#pragma unroll
  for (int q = 0; q < kQA; ++q)
    *reinterpret_cast<u32x4*>(As + (tid / kKChunks + kRowStep * q) * kLdsRow + kc * 8) = st.a[q];
#pragma unroll
  for (int q = 0; q < kQB; ++q)
    *reinterpret_cast<u32x4*>(Bs + (tid / kKChunks + kRowStep * q) * kLdsRow + kc * 8) = st.b[q];
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

template <int ACT>
__global__ __launch_bounds__(kThreads) void linear_act_fwd_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, uint32_t* __restrict__ codes,
    uint16_t* __restrict__ z, int64_t M, int64_t N, int64_t K) {
  using A = ActOf<ACT>;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int wm = wave / kWN, wn = wave % kWN;

  int64_t tm, tn;
  block_tile((M + kBM - 1) / kBM, (N + kBN - 1) / kBN, tm, tn);
  const int64_t m0 = tm * kBM, n0 = tn * kBN;

  f32x16 acc[kTM][kTN];
#pragma unroll
  for (int i = 0; i < kTM; ++i)
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int64_t kt_count = (K + kBK - 1) / kBK;
  const Operands op = make_operands(x, w, m0, n0, M, N, K);

#if LMBP_LIN_DIRECT
  // Direct path. A stage holds the A tile (BM rows) then the B tile (BN rows), each
  // row 32 bf16 = four 16-byte units; unit u of row r holds k-chunk u ^ ((r >> 2) & 3),
  // so that the operand reads of 16 consecutive rows at one k-chunk hit 16 distinct
  // bank groups. One load instruction of a wave fills 1 KiB (16 rows): lane l writes
  // unit l % 4 of row l / 4, i.e. fetches k-chunk (l % 4) ^ ((row >> 2) & 3) of that
  // row (each row's four lanes read its 64 contiguous bytes in permuted order).
  constexpr int kWaves = kWM * kWN;
  constexpr int kBlocksA = kBM / 16, kBlocksB = kBN / 16;
  static_assert(kBlocksA % kWaves == 0 && kBlocksB % kWaves == 0, "load blocks per wave");
  constexpr int kLA = kBlocksA / kWaves, kLB = kBlocksB / kWaves;
  constexpr int kLoadsPerStage = kLA + kLB;
  typedef __attribute__((address_space(3))) void lds_void;
  uint32_t ld_a[kLA], ld_b[kLB];  // byte offset in the operand (row start + chunk), k step 0
  {
    const int r_in = lane >> 2;
    const int kc = (lane & 3) ^ ((r_in >> 2) & 3);   // block rows start at multiples of 16
#pragma unroll
    for (int q = 0; q < kLA; ++q)
      ld_a[q] = uint32_t(((wave + kWaves * q) * 16 + r_in) * K * 2 + kc * 16);
#pragma unroll
    for (int q = 0; q < kLB; ++q)
      ld_b[q] = uint32_t(((wave + kWaves * q) * 16 + r_in) * K * 2 + kc * 16);
  }
  const uint32_t kc_bytes = uint32_t(((lane & 3) ^ (((lane >> 2) >> 2) & 3)) * 16);
  auto issue_stage = [&](int64_t kt) {
    uint16_t* S = lds + int(kt % kStages) * kDStageElems;
    const uint32_t k0b = uint32_t(kt * kBK * 2);
    const bool kin = kt * kBK + int64_t(kc_bytes / 2) < K;
#pragma unroll
    for (int q = 0; q < kLA; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          op.x, (lds_void*)(S + (wave + kWaves * q) * 16 * kBK), 16,
          kin ? ld_a[q] + k0b : kOutOfRange, 0, 0, 0);
#pragma unroll
    for (int q = 0; q < kLB; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          op.w, (lds_void*)(S + kBM * kBK + (wave + kWaves * q) * 16 * kBK), 16,
          kin ? ld_b[q] + k0b : kOutOfRange, 0, 0, 0);
  };
  // Operand reads: lane l reads row (base + l % 32), k-chunk 2 kk + l / 32.
  const int swz = ((lane & 31) >> 2) & 3;   // (row >> 2) & 3; wave rows start at multiples of 32
  int a_row[kTM], b_row[kTN];
#pragma unroll
  for (int i = 0; i < kTM; ++i) a_row[i] = (wm * kTM * 32 + i * 32 + (lane & 31)) * kBK;
#pragma unroll
  for (int j = 0; j < kTN; ++j) b_row[j] = kBM * kBK + (wn * kTN * 32 + j * 32 + (lane & 31)) * kBK;
  auto compute = [&](const uint16_t* S) {
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int unit = ((2 * kk + (lane >> 5)) ^ swz) * 8;
      bf16x8 a[kTM], b[kTN];
#pragma unroll
      for (int i = 0; i < kTM; ++i) a[i] = *reinterpret_cast<const bf16x8*>(S + a_row[i] + unit);
#pragma unroll
      for (int j = 0; j < kTN; ++j) b[j] = *reinterpret_cast<const bf16x8*>(S + b_row[j] + unit);
#pragma unroll
      for (int i = 0; i < kTM; ++i)
#pragma unroll
        for (int j = 0; j < kTN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };
  // Wait until at most `pending` stages of this wave's loads are outstanding (the
  // vector-memory counter counts the direct loads; nothing else uses it in the loop).
  auto wait_stages = [&](int64_t pending) {
    static_assert(kStages - 2 <= 3, "wait table");
    if (pending <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else if (pending == 1) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(kLoadsPerStage) : "memory");
    else if (pending == 2) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(2 * kLoadsPerStage) : "memory");
    else asm volatile("s_waitcnt vmcnt(%0)" :: "n"(3 * kLoadsPerStage) : "memory");
  };
  for (int s = 0; s < kStages - 1; ++s)
    if (s < kt_count) issue_stage(s);
  for (int64_t kt = 0; kt < kt_count; ++kt) {
    const int64_t issued_after = (kt_count - 1 - kt < kStages - 2) ? kt_count - 1 - kt : kStages - 2;
    wait_stages(issued_after);
    asm volatile("s_barrier" ::: "memory");   // every wave's loads of step kt are in LDS
    if (kt + kStages - 1 < kt_count) issue_stage(kt + kStages - 1);   // into step kt - 1's buffer
    compute(lds + int(kt % kStages) * kDStageElems);
  }
  __syncthreads();
#else
  // Operand read offsets (in bf16 elements) inside one stage.
  const int a_off = (wm * kTM * 32 + (lane & 31)) * kLdsRow + 8 * (lane >> 5);
  const int b_off = kAElems + (wn * kTN * 32 + (lane & 31)) * kLdsRow + 8 * (lane >> 5);

  auto compute = [&](const uint16_t* S) {
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8 a[kTM], b[kTN];
#pragma unroll
      for (int i = 0; i < kTM; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(S + a_off + i * 32 * kLdsRow + kk * 16);
#pragma unroll
      for (int j = 0; j < kTN; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(S + b_off + j * 32 * kLdsRow + kk * 16);
#pragma unroll
      for (int i = 0; i < kTM; ++i)
#pragma unroll
        for (int j = 0; j < kTN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };
  auto stage_ptr = [&](int64_t kt) { return lds + int(kt & 1) * kStageElems; };

#if LMBP_LIN_PREFETCH == 2
  // Two register stages: the loads of step kt + 2 are issued before the MFMAs of step
  // kt, so they have two steps of MFMA work to arrive before they are written to LDS.
  Stage s0, s1;
  if (kt_count > 0) load_stage(s0, op, K, 0);
  if (kt_count > 1) load_stage(s1, op, K, kBK);
  if (kt_count > 0) store_stage(s0, lds, lds + kAElems);
  __syncthreads();
  auto step = [&](int64_t kt, Stage& free_regs, Stage& next_regs) {
    if (kt + 2 < kt_count) load_stage(free_regs, op, K, (kt + 2) * kBK);
    compute(stage_ptr(kt));
    if (kt + 1 < kt_count) {
      uint16_t* D = stage_ptr(kt + 1);
      store_stage(next_regs, D, D + kAElems);
    }
    __syncthreads();
  };
  for (int64_t kt = 0; kt < kt_count; kt += 2) {
    step(kt, s0, s1);
    if (kt + 1 < kt_count) step(kt + 1, s1, s0);
  }
#else
  // One register stage: the loads of step kt + 1 are in flight during the MFMAs of kt.
  Stage st;
  if (kt_count > 0) {
    load_stage(st, op, K, 0);
    store_stage(st, lds, lds + kAElems);
  }
  __syncthreads();
  for (int64_t kt = 0; kt < kt_count; ++kt) {
    const bool more = kt + 1 < kt_count;
    if (more) load_stage(st, op, K, (kt + 1) * kBK);
    compute(stage_ptr(kt));
    if (more) {
      uint16_t* D = stage_ptr(kt + 1);
      store_stage(st, D, D + kAElems);
    }
    __syncthreads();
  }
#endif
#endif  // LMBP_LIN_DIRECT

  // Epilogue, part 1: bias, rounding to bf16, the tile into LDS (row-major, padded).
  uint16_t* E = lds;
#pragma unroll
  for (int j = 0; j < kTN; ++j) {
    const int col = wn * kTN * 32 + j * 32 + (lane & 31);
    const float bj = (bias != nullptr && n0 + col < N)
                         ? __uint_as_float(uint32_t(bias[n0 + col]) << 16) : 0.0f;
#pragma unroll
    for (int i = 0; i < kTM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * kTM * 32 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        E[row * kEpiRow + col] = uint16_t(pack_bf16x2(acc[i][j][r] + bj, 0.0f) & 0xffffu);
      }
  }
  __syncthreads();

  // Part 2: thread owns columns c16 .. c16 + 15 of rows tid / (BN/16) + step * g.
  const int c16 = (tid % kEpiThreadsPerRow) * 16;
  if (n0 + c16 >= N) return;  // N is a multiple of 16: a group is wholly in or out
#pragma unroll 2
  for (int row = tid / kEpiThreadsPerRow; row < kBM; row += kEpiRowStep) {
    if (m0 + row >= M) break;
    const u32x4 v0 = *reinterpret_cast<const u32x4*>(E + row * kEpiRow + c16);
    const u32x4 v1 = *reinterpret_cast<const u32x4*>(E + row * kEpiRow + c16 + 8);
    float f0[8], f1[8], o0[8], o1[8];
    BF16::unpack(v0, f0);
    BF16::unpack(v1, f1);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      o0[e] = act_value<ACT, false>(f0[e]);
      o1[e] = act_value<ACT, false>(f1[e]);
    }
    const int64_t base = (m0 + row) * N + n0 + c16;   // flat element index, multiple of 16
    *reinterpret_cast<u32x4*>(y + base) = BF16::pack(o0);
    *reinterpret_cast<u32x4*>(y + base + 8) = BF16::pack(o1);
    codes[base / 16] = codes_of<A>(f0) | (codes_of<A>(f1) << 16);
    if (z != nullptr) {
      *reinterpret_cast<u32x4*>(z + base) = v0;
      *reinterpret_cast<u32x4*>(z + base + 8) = v1;
    }
  }
}

}  // namespace

hipError_t launch_linear_act_fwd(int act, int64_t M, int64_t N, int64_t K, const void* x,
                                 const void* w, const void* bias, void* y, uint32_t* codes,
                                 void* z, hipStream_t s) {
  const int64_t blocks = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  auto* xp = static_cast<const uint16_t*>(x);
  auto* wp = static_cast<const uint16_t*>(w);
  auto* bp = static_cast<const uint16_t*>(bias);
  auto* yp = static_cast<uint16_t*>(y);
  auto* zp = static_cast<uint16_t*>(z);
  const size_t lds = size_t(kLdsElems) * 2;
  auto kern = act == kGelu ? linear_act_fwd_kernel<kGelu> : linear_act_fwd_kernel<kSilu>;
  // More than 64 KiB of dynamic LDS must be allowed explicitly (once per kernel).
  static hipError_t attr_gelu = hipFuncSetAttribute(
      reinterpret_cast<const void*>(linear_act_fwd_kernel<kGelu>),
      hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  static hipError_t attr_silu = hipFuncSetAttribute(
      reinterpret_cast<const void*>(linear_act_fwd_kernel<kSilu>),
      hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  const hipError_t attr = act == kGelu ? attr_gelu : attr_silu;
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kern, dim3(unsigned(blocks)), dim3(kThreads), lds, s, xp, wp, bp, yp, codes,
                     zp, M, N, K);
  return hipGetLastError();
}

}  // namespace lmbp
