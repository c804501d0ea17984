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
// Tiling: a 256-thread block computes a 128 x 128 tile of z, each of its four waves a
// 64 x 64 quarter as 2 x 2 MFMA tiles of 32 x 32. K advances in steps of 64 through
// two LDS buffers per operand; the global loads of the next step are in flight while
// the MFMAs of the current one run. LDS rows are padded to 144 bytes so that the
// 16-byte operand reads of 32 consecutive rows fall on distinct banks. Lane layout of
// the MFMA (checked on the hardware): lane l supplies row l % 32 of A and column l % 32
// of B at k = 8 (l / 32) .. + 7, and holds result rows 8 (r / 4) + 4 (l / 32) + r % 4
// of column l % 32 in accumulator register r.
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

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kThreads = 256;
constexpr int kLdsRow = kBK + 8;                  // bf16 per operand row in LDS (144 bytes)
constexpr int kOpElems = kBM * kLdsRow;           // one operand buffer
constexpr int kEpiRow = kBN + 8;                  // bf16 per row of the epilogue tile (272 bytes)
constexpr int kLdsBytes = 2 * 2 * kOpElems * 2;   // two stages of A and B
static_assert(kBM * kEpiRow * 2 <= kLdsBytes, "epilogue tile must fit in the operand buffers");
static_assert(kBM == kBN, "the load mapping assumes square tiles");
constexpr int kXcds = 8;
constexpr int kGroupM = 8;

// One K step of both operands, 16-byte chunks: chunk c = tid + 256 q (q < 4) is row
// c / 8, k-chunk c % 8 of the 128 x 64 tile. Rows at or beyond `rows` and k beyond K
// load zeros (K is a multiple of 8, so a chunk is wholly inside or outside).
struct Stage {
  u32x4 a[4], b[4];
};

__device__ inline void load_stage(Stage& st, const uint16_t* __restrict__ x,
                                  const uint16_t* __restrict__ w, int64_t m0, int64_t n0,
                                  int64_t M, int64_t N, int64_t K, int64_t k0) {
  const int tid = threadIdx.x;
  const int kc = tid & 7;
  const int64_t k = k0 + kc * 8;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int row = (tid >> 3) + 32 * q;
    const bool kin = k < K;
    st.a[q] = (kin && m0 + row < M) ? *reinterpret_cast<const u32x4*>(x + (m0 + row) * K + k)
                                    : u32x4{0u, 0u, 0u, 0u};
    st.b[q] = (kin && n0 + row < N) ? *reinterpret_cast<const u32x4*>(w + (n0 + row) * K + k)
                                    : u32x4{0u, 0u, 0u, 0u};
  }
}

__device__ inline void store_stage(const Stage& st, uint16_t* As, uint16_t* Bs) {
  const int tid = threadIdx.x;
  const int kc = tid & 7;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int row = (tid >> 3) + 32 * q;
    *reinterpret_cast<u32x4*>(As + row * kLdsRow + kc * 8) = st.a[q];
    *reinterpret_cast<u32x4*>(Bs + row * kLdsRow + kc * 8) = st.b[q];
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

template <int ACT>
__global__ __launch_bounds__(kThreads) void linear_act_fwd_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, uint32_t* __restrict__ codes,
    uint16_t* __restrict__ z, int64_t M, int64_t N, int64_t K) {
  using A = ActOf<ACT>;
  __shared__ __attribute__((aligned(16))) uint16_t lds[kLdsBytes / 2];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int wm = wave >> 1, wn = wave & 1;

  int64_t tm, tn;
  block_tile((M + kBM - 1) / kBM, (N + kBN - 1) / kBN, tm, tn);
  const int64_t m0 = tm * kBM, n0 = tn * kBN;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int64_t kt_count = (K + kBK - 1) / kBK;
  Stage st;
  if (kt_count > 0) {
    load_stage(st, x, w, m0, n0, M, N, K, 0);
    store_stage(st, lds, lds + 2 * kOpElems);
  }
  __syncthreads();

  // Operand read offsets (in bf16 elements) inside one buffer.
  const int a_off = (wm * 64 + (lane & 31)) * kLdsRow + 8 * (lane >> 5);
  const int b_off = (wn * 64 + (lane & 31)) * kLdsRow + 8 * (lane >> 5);

  for (int64_t kt = 0; kt < kt_count; ++kt) {
    const int cur = int(kt & 1);
    const bool more = kt + 1 < kt_count;
    if (more) load_stage(st, x, w, m0, n0, M, N, K, (kt + 1) * kBK);
    const uint16_t* As = lds + cur * kOpElems;
    const uint16_t* Bs = lds + (2 + cur) * kOpElems;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(As + a_off + i * 32 * kLdsRow + kk * 16);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(Bs + b_off + j * 32 * kLdsRow + kk * 16);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (more) store_stage(st, lds + (1 - cur) * kOpElems, lds + (3 - cur) * kOpElems);
    __syncthreads();
  }

  // Epilogue, part 1: bias, rounding to bf16, the tile into LDS (row-major, padded).
  uint16_t* E = lds;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int col = wn * 64 + j * 32 + (lane & 31);
    const float bj = (bias != nullptr && n0 + col < N)
                         ? __uint_as_float(uint32_t(bias[n0 + col]) << 16) : 0.0f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        E[row * kEpiRow + col] = uint16_t(pack_bf16x2(acc[i][j][r] + bj, 0.0f) & 0xffffu);
      }
  }
  __syncthreads();

  // Part 2: thread owns columns c16 .. c16 + 15 of rows (tid / 8) + 32 g.
  const int c16 = (tid & 7) * 16;
  if (n0 + c16 >= N) return;  // N is a multiple of 16: a group is wholly in or out
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int row = (tid >> 3) + 32 * g;
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
  if (act == kGelu)
    hipLaunchKernelGGL(linear_act_fwd_kernel<kGelu>, dim3(unsigned(blocks)), dim3(kThreads), 0, s,
                       xp, wp, bp, yp, codes, zp, M, N, K);
  else
    hipLaunchKernelGGL(linear_act_fwd_kernel<kSilu>, dim3(unsigned(blocks)), dim3(kThreads), 0, s,
                       xp, wp, bp, yp, codes, zp, M, N, K);
  return hipGetLastError();
}

}  // namespace lmbp
