// bf16 MFMA GEMM for gfx950: C[M, N] = A[M, K] . W[N, K]^T with fp32 accumulation.
//
// Both operands are K-contiguous (activations [M, K], weights [out, in]), so every
// global load and every LDS fragment read is a 16-byte vector along K.  A workgroup
// of WAVES_M x WAVES_N wavefronts owns a BM x BN tile; each wavefront owns
// TM x TN blocks of 32 x 32 computed with v_mfma_f32_32x32x16_bf16.
//
// Pipeline: two BK-slices are in flight in registers while a third is multiplied out
// of LDS (two LDS buffers, one barrier per slice), so a slice's global loads have two
// slices of MFMA work to arrive.  LDS rows are padded by 16 bytes so the 32 lanes that
// read one fragment column hit distinct banks.
//
// Split-K (for outputs with too few tiles to fill the chip): split s of a tile
// accumulates K-slices [s*nk, (s+1)*nk), stores its fp32 partial tile to a workspace,
// and takes a ticket on the tile; the last split to arrive adds the partials in split
// order (0, 1, ..., S-1), so the result does not depend on arrival order, runs the
// epilogue and resets the ticket.
//
// Epilogues:  EPI_BF16    C = bf16((acc + bias[n]) * scale)
//             EPI_ADD_F32 C(fp32) += acc            (residual stream update)
//             EPI_SWIGLU  weights interleave gate/up rows in groups of 32, so a
//                         wavefront's two 32-column blocks hold gate and up of the
//                         same outputs: C = bf16(silu(g) * u), ldc over ffn columns.
// Requirements: K % (64 * splits) == 0; M, N arbitrary (tails clamped on load, masked
// on store).
#include "common.hpp"
#include "internal.hpp"

namespace cora {

constexpr int BK = 64;
constexpr int LDK = BK + 8;  // padded LDS row, in bf16 elements

// n 16-byte loads at byte offset voff + i * step (step uniform) through a buffer resource
template <int N>
__device__ __forceinline__ void buf_load(u32x4_t (&r)[N], __amdgpu_buffer_rsrc_t rs, int voff,
                                         int step) {
#pragma unroll
  for (int i = 0; i < N; ++i)
    r[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, i * step, 0));
}

template <int WAVES_M, int WAVES_N, int TM, int TN, int EPI>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64) void k_gemm(GemmArgs g) {
  constexpr int NT = WAVES_M * WAVES_N * 64;
  constexpr int BM = WAVES_M * TM * 32, BN = WAVES_N * TN * 32;
  constexpr int CA = BM * BK / 8 / NT;  // 16-byte chunks per thread per slice
  constexpr int CB = BN * BK / 8 / NT;
  constexpr int NACC = TM * TN * 16;    // accumulators per thread
  static_assert(CA * NT * 8 == BM * BK && CB * NT * 8 == BN * BK, "tile/thread mismatch");
  static_assert(EPI != EPI_SWIGLU || TN == 2, "SwiGLU epilogue pairs two 32-column blocks");

  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDK];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int num_m = (g.M + BM - 1) / BM;
  const int li = xcd_remap(blockIdx.x, gridDim.x);
  const int split = li % g.splits, tile = li / g.splits;
  const int tile_m = tile % num_m, tile_n = tile / num_m;
  const int m0 = tile_m * BM, n0 = tile_n * BN;
  const int nk = g.K / BK / g.splits;
  const int64_t k_base = (int64_t)split * nk * BK;

  // operands through buffer resources: 32-bit byte offsets, and rows past M or N read
  // as zero (hardware range check), so tails need no clamping
  const int64_t a_bytes = (int64_t)g.M * g.lda * 2, b_bytes = (int64_t)g.N * g.ldw * 2;
  const __amdgpu_buffer_rsrc_t a_rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)g.A, (short)0, (int)(a_bytes > 0xffffffffLL ? 0xffffffffu : (uint32_t)a_bytes),
      0x00020000);
  const __amdgpu_buffer_rsrc_t b_rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)g.W, (short)0, (int)(b_bytes > 0xffffffffLL ? 0xffffffffu : (uint32_t)b_bytes),
      0x00020000);
  const int c_r = tid >> 3, c_k = (tid & 7) * 8;
  const int a_off = (int)(((int64_t)(m0 + c_r) * g.lda + k_base + c_k) * 2);
  const int b_off = (int)(((int64_t)(n0 + c_r) * g.ldw + k_base + c_k) * 2);
  const int a_step = (NT / 8) * (int)g.lda * 2;  // next chunk of this thread: NT/8 rows down
  const int b_step = (NT / 8) * (int)g.ldw * 2;
  const int lds_off = c_r * LDK + c_k;
  constexpr int LDS_STEP = (NT / 8) * LDK;

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  u32x4_t ra0[CA], rb0[CB], ra1[CA], rb1[CB];
#define GEMM_FETCH(ra, rb, kt)                                   \
  do {                                                           \
    buf_load<CA>(ra, a_rs, a_off + (kt) * BK * 2, a_step);       \
    buf_load<CB>(rb, b_rs, b_off + (kt) * BK * 2, b_step);       \
  } while (0)
  auto stash = [&](int buf, const u32x4_t(&ra)[CA], const u32x4_t(&rb)[CB]) {
#pragma unroll
    for (int i = 0; i < CA; ++i)
      *reinterpret_cast<u32x4_t*>(&As[buf][lds_off + i * LDS_STEP]) = ra[i];
#pragma unroll
    for (int i = 0; i < CB; ++i)
      *reinterpret_cast<u32x4_t*>(&Bs[buf][lds_off + i * LDS_STEP]) = rb[i];
  };

  // fragment read offsets: lane holds row (lane % 32), k half (lane / 32) * 8
  const int frag_r = lane & 31, frag_k = (lane >> 5) * 8;
  const int a_base = (wm * TM * 32 + frag_r) * LDK + frag_k;
  const int b_base = (wn * TN * 32 + frag_r) * LDK + frag_k;
  // fragments of step kk+16 are read while the MFMAs of step kk run; scheduling
  // barriers keep the compiler from hoisting a whole slice's reads (register pressure)
  auto load_frags = [&](int buf, int kk, bf16x8_t(&fa)[TM], bf16x8_t(&fb)[TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
      fa[i] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(&As[buf][a_base + i * 32 * LDK + kk]));
#pragma unroll
    for (int j = 0; j < TN; ++j)
      fb[j] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(&Bs[buf][b_base + j * 32 * LDK + kk]));
  };
  auto mfmas = [&](const bf16x8_t(&fa)[TM], const bf16x8_t(&fb)[TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  };
  auto compute = [&](int buf) {
    bf16x8_t fa0[TM], fb0[TN], fa1[TM], fb1[TN];
    load_frags(buf, 0, fa0, fb0);
    load_frags(buf, 16, fa1, fb1);
    mfmas(fa0, fb0);
    __builtin_amdgcn_sched_barrier(0);
    load_frags(buf, 32, fa0, fb0);
    mfmas(fa1, fb1);
    __builtin_amdgcn_sched_barrier(0);
    load_frags(buf, 48, fa1, fb1);
    mfmas(fa0, fb0);
    __builtin_amdgcn_sched_barrier(0);
    mfmas(fa1, fb1);
  };

  // slices kt (LDS), kt+1 and kt+2 (registers) in flight
  GEMM_FETCH(ra0, rb0, 0);
  if (nk > 1) GEMM_FETCH(ra1, rb1, 1);
  stash(0, ra0, rb0);
  __syncthreads();
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    if (kt + 2 < nk) GEMM_FETCH(ra0, rb0, kt + 2);
    compute(0);
    stash(1, ra1, rb1);
    __syncthreads();
    if (kt + 3 < nk) GEMM_FETCH(ra1, rb1, kt + 3);
    compute(1);
    if (kt + 2 < nk) stash(0, ra0, rb0);
    __syncthreads();
  }
  if (kt < nk) compute(0);  // odd slice count: the last slice sits in buffer 0
#undef GEMM_FETCH
  if (g.splits > 1) {
    // deterministic split-K: partials laid out [tile][split][thread][NACC]
    float* part = g.ws + ((int64_t)tile * g.splits) * NT * NACC;
    float* mine = part + ((int64_t)split * NT + tid) * NACC;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; e += 4)
          *reinterpret_cast<f32x4_t*>(mine + (i * TN + j) * 16 + e) =
              f32x4_t{acc[i][j][e], acc[i][j][e + 1], acc[i][j][e + 2], acc[i][j][e + 3]};
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = atomicAdd(&g.counters[tile], 1) == g.splits - 1;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    for (int s = 0; s < g.splits; ++s) {
      const float* p = part + ((int64_t)s * NT + tid) * NACC;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; e += 4) {
            const f32x4_t v = *reinterpret_cast<const f32x4_t*>(p + (i * TN + j) * 16 + e);
            acc[i][j][e] += v[0];
            acc[i][j][e + 1] += v[1];
            acc[i][j][e + 2] += v[2];
            acc[i][j][e + 3] += v[3];
          }
    }
    if (tid == 0) g.counters[tile] = 0;
  }

  // epilogue: acc[i][j][e] is C[row, col] with
  //   row = m0 + wm*TM*32 + i*32 + 8*(e/4) + 4*(lane/32) + e%4,  col = n0 + wn*TN*32 + j*32 + lane%32
  const int col_l = lane & 31, row_q = (lane >> 5) * 4;
  if constexpr (EPI == EPI_SWIGLU) {
    const int jcol = (n0 + wn * 64) / 2 + col_l;  // output (ffn) column
    if (2 * (jcol - col_l) < g.N) {
      uint16_t* C = reinterpret_cast<uint16_t*>(g.C);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * TM * 32 + i * 32 + 8 * (e >> 2) + row_q + (e & 3);
          if (row < g.M) {
            const float gt = acc[i][0][e], up = acc[i][1][e];
            const float s = gt / (1.0f + __expf(-gt));
            C[(int64_t)row * g.ldc + jcol] = (uint16_t)f32_to_bf16_bits(s * up);
          }
        }
    }
  } else {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * TN * 32 + j * 32 + col_l;
      if (col >= g.N) continue;
      const float bias = (EPI == EPI_BF16 && g.bias) ? g.bias[col] : 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * TM * 32 + i * 32 + 8 * (e >> 2) + row_q + (e & 3);
          if (row >= g.M) continue;
          if constexpr (EPI == EPI_ADD_F32) {
            float* C = reinterpret_cast<float*>(g.C);
            C[(int64_t)row * g.ldc + col] += acc[i][j][e];
          } else {
            uint16_t* C = reinterpret_cast<uint16_t*>(g.C);
            C[(int64_t)row * g.ldc + col] =
                (uint16_t)f32_to_bf16_bits((acc[i][j][e] + bias) * g.scale);
          }
        }
    }
  }
}

// ---- tile configurations -------------------------------------------------------------
enum GemmCfg { CFG_BIG = 0, CFG_SMALL_M = 1 };

static void cfg_tile(int cfg, int epi, int* bm, int* bn) {
  if (cfg == CFG_SMALL_M) { *bm = 32; *bn = epi == EPI_SWIGLU ? 128 : 128; return; }
  *bm = 256; *bn = 128;
}

GemmPlan gemm_plan(int epi, int M, int N, int K, int num_cus) {
  GemmPlan p{};
  p.cfg = M <= 64 ? CFG_SMALL_M : CFG_BIG;
  int bm, bn;
  cfg_tile(p.cfg, epi, &bm, &bn);
  p.tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  p.splits = 1;
  if (epi == EPI_ADD_F32 && p.cfg == CFG_BIG) {
    // split the K loop until the grid covers the chip, keeping >= 8 slices per split
    const int nk = K / BK;
    while (p.tiles * p.splits < num_cus && p.splits < 8 && nk % (p.splits * 2) == 0 &&
           nk / (p.splits * 2) >= 8)
      p.splits *= 2;
  }
  const int nt = p.cfg == CFG_SMALL_M ? 256 : 256;
  p.ws_floats = p.splits > 1 ? (size_t)p.tiles * p.splits * bm * bn : 0;
  (void)nt;
  return p;
}

template <int WAVES_M, int WAVES_N, int TM, int TN, int EPI>
static hipError_t run(const GemmArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL((k_gemm<WAVES_M, WAVES_N, TM, TN, EPI>), dim3(grid),
                     dim3(WAVES_M * WAVES_N * 64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm(int epi, const GemmArgs& in, const GemmPlan& p, hipStream_t s) {
  if (in.M == 0 || in.N == 0) return hipSuccess;
  if (in.K % (BK * p.splits) != 0) return hipErrorInvalidValue;
  if (p.splits > 1 && (!in.ws || !in.counters)) return hipErrorInvalidValue;
  GemmArgs a = in;
  a.splits = p.splits;
  const int grid = p.tiles * p.splits;
  const bool small = p.cfg == CFG_SMALL_M;
  switch (epi) {
    case EPI_BF16:
      return small ? run<1, 4, 1, 1, EPI_BF16>(a, grid, s) : run<2, 2, 4, 2, EPI_BF16>(a, grid, s);
    case EPI_ADD_F32:
      return small ? run<1, 4, 1, 1, EPI_ADD_F32>(a, grid, s)
                   : run<2, 2, 4, 2, EPI_ADD_F32>(a, grid, s);
    case EPI_SWIGLU:
      return small ? run<1, 2, 1, 2, EPI_SWIGLU>(a, grid, s)
                   : run<2, 2, 4, 2, EPI_SWIGLU>(a, grid, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace cora
