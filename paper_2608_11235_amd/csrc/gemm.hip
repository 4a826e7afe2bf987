// bf16 MFMA GEMM for gfx950: C[M, N] = A[M, K] . W[N, K]^T with fp32 accumulation.
//
// Both operands are K-contiguous (activations [M, K], weights [out, in]), so every
// global load and every LDS fragment read is a 16-byte vector along K.  A workgroup
// of WAVES_M x WAVES_N wavefronts owns a BM x BN tile; each wavefront owns
// TM x TN blocks of 32 x 32 computed with v_mfma_f32_32x32x16_bf16.
//
// Pipelines (template parameter PIPE), all with two LDS buffers and one barrier per BK-slice:
//   PIPE 0  slice kt+1 in registers while slice kt is multiplied out of LDS; fragments of
//           k-step s+16 read during the MFMAs of step s (16-wave config: no registers
//           left for a second stage).
//   PIPE 1  slices kt+1 and kt+2 in registers, plain order (small-M config).
//   PIPE 2  slices kt+1 and kt+2 in registers, and the slice loop body is branch-free so
//           the scheduler can interleave everything: the LDS stash of slice kt+1 and the
//           global fetch of slice kt+3 are spread over the MFMA steps of slice kt (MFMA /
//           ds_read / ds_write / buffer_load groups), and the barrier sits before the last
//           MFMA group, which then covers the first fragment reads of the next slice.
//           Every thread stores all its chunks (rows past the tile land in spare LDS rows)
//           and the fetch index is clamped, so nothing in the loop is conditional.  Memory
//           and MFMA work overlap instead of alternating; on the 512 x 24576 x 4096
//           gate/up GEMM this takes the 12-wave config from 113 to 90 us.
// LDS rows are padded by 16 bytes so the lanes that read one fragment column hit distinct
// banks.
//
// Split-K (for outputs with too few tiles to fill the chip): split s of a tile
// accumulates K-slices [s*nk, (s+1)*nk) and stores its fp32 partial tile (EPI_PART_F32);
// a row-wise kernel downstream adds the partials in split order, so results do not depend
// on scheduling, and applies what the output needs next (residual add + RMSNorm, or bias +
// RoPE + head layout for q/k/v).
//
// Epilogues:  EPI_BF16    C = bf16((acc + bias[n]) * scale)
//             EPI_ADD_F32 C(fp32) += acc            (residual stream update)
//             EPI_PART_F32  split s stores acc to its own fp32 slab of C
//             EPI_SWIGLU  weights interleave gate/up rows in groups of 32, so a
//                         wavefront's two 32-column blocks hold gate and up of the
//                         same outputs: C = bf16(silu(g) * u), ldc over ffn columns.
//             EPI_QKV_ROPE  bias, rotate-half RoPE on q and k, head-major q/k and
//                         transposed v written straight from the accumulators.
//             EPI_TOP1    no C: per row and wavefront column range, (max, first arg max,
//                         sum of exp) of the bf16 logits EPI_BF16 would store (Eq. 1).
// Weights are either row-major or stored in 64 x 64 blocks (w_packed), in which case a
// tile's BK-slice of W is a run of whole 8 KB blocks.
// Requirements: K % (64 * splits) == 0; M, N arbitrary (tails clamped on load, masked
// on store).
#include <hip/hip_ext.h>
#include <limits.h>

#include "common.hpp"
#include "internal.hpp"

namespace cora {

constexpr int BK = 64;
constexpr int LDK = BK + 8;  // padded LDS row, in bf16 elements

// N 16-byte loads at byte offsets voff + i * step (step uniform) through a buffer resource,
// the last one from its own per-lane offset voff_last (an offset past the resource's range
// makes the hardware return zeros without touching memory)
template <int N>
__device__ __forceinline__ void buf_load_tail(u32x4_t (&r)[N], __amdgpu_buffer_rsrc_t rs, int voff,
                                              int voff_last, int step) {
#pragma unroll
  for (int i = 0; i < N; ++i)
    r[i] = __builtin_bit_cast(
        u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, i + 1 < N ? voff : voff_last, i * step, 0));
}

// N 16-byte loads at per-chunk byte offsets voff[i] + koff (koff uniform); when the chunks
// do not divide evenly and EXACT is false, the last one only where last_ok
template <int N, bool EXACT>
__device__ __forceinline__ void buf_load_chunks(u32x4_t (&r)[N], __amdgpu_buffer_rsrc_t rs,
                                                const int (&voff)[N], int koff, bool last_ok) {
#pragma unroll
  for (int i = 0; i < N; ++i)
    if (EXACT || i + 1 < N || last_ok)
      r[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, voff[i] + koff, 0, 0));
}

// N 16-byte loads at byte offsets voff + i * step (step uniform); when the chunks do not
// divide evenly and EXACT is false, the last one only where last_ok
template <int N, bool EXACT>
__device__ __forceinline__ void buf_load(u32x4_t (&r)[N], __amdgpu_buffer_rsrc_t rs, int voff,
                                         int step, bool last_ok) {
#pragma unroll
  for (int i = 0; i < N; ++i)
    if (EXACT || i + 1 < N || last_ok)
      r[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, i * step, 0));
}

template <int WAVES_M, int WAVES_N, int TM, int TN, int EPI, int PIPE>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64) void k_gemm(GemmArgs g) {
  constexpr int NT = WAVES_M * WAVES_N * 64;
  constexpr int BM = WAVES_M * TM * 32, BN = WAVES_N * TN * 32;
  constexpr int CA = (BM * BK / 8 + NT - 1) / NT;  // 16-byte chunks per thread per slice
  constexpr int CB = (BN * BK / 8 + NT - 1) / NT;
  constexpr bool A_EXACT = CA * NT * 8 == BM * BK, B_EXACT = CB * NT * 8 == BN * BK;
  constexpr int NACC = TM * TN * 16;    // accumulators per thread
  static_assert(NT % 8 == 0, "threads must cover whole 64-element rows");
  static_assert(EPI != EPI_SWIGLU || TN % 2 == 0, "SwiGLU epilogue pairs 32-column blocks");
  static_assert(PIPE != 2 || TM * TN == 4 || TM * TN == 2, "PIPE 2 schedules 4 or 2 MFMAs per k-step");

  // PIPE 2 stores every thread's chunks unconditionally: rows past the tile land in spare
  // LDS rows (CA * NT / 8 >= BM)
  constexpr int A_ROWS = PIPE == 2 ? CA * NT / 8 : BM, B_ROWS = PIPE == 2 ? CB * NT / 8 : BN;
  // one LDS array: the operand buffers As [2][A_ROWS * LDK] then Bs [2][B_ROWS * LDK]; the
  // epilogues reuse it whole
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * (A_ROWS + B_ROWS) * LDK];
  auto As = reinterpret_cast<uint16_t(*)[A_ROWS * LDK]>(lds);
  auto Bs = reinterpret_cast<uint16_t(*)[B_ROWS * LDK]>(lds + 2 * A_ROWS * LDK);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int num_m = (g.M + BM - 1) / BM;
  // logical order: split-major, then N tile, then M tile.  xcd_remap hands each XCD a
  // contiguous run of that order, so an XCD's workgroups share one K range (its L2 holds
  // only that range of A) and, within it, the M tiles of a run of N tiles (each weight
  // byte is fetched by one XCD).
  const int li = xcd_remap(blockIdx.x, gridDim.x);
  const int n_tiles = gridDim.x / g.splits;
  const int split = li / n_tiles, tile = li - split * n_tiles;
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
  const int b_off = (int)(((int64_t)(n0 + c_r) * g.ldw + k_base + c_k) * 2);  // row-major
  const int a_step = (NT / 8) * (int)g.lda * 2;  // next chunk of this thread: NT/8 rows down
  const int b_step = (NT / 8) * (int)g.ldw * 2;
  const int lds_off = c_r * LDK + c_k;
  constexpr int LDS_STEP = (NT / 8) * LDK;
  const bool a_last = tid + (CA - 1) * NT < BM * BK / 8;
  const bool b_last = tid + (CB - 1) * NT < BN * BK / 8;
  // B chunk i of slice kt sits at byte b_chunk[i] + kt * b_kstride: row-major weights (row
  // c_r + i NT / 8 of the tile, next slice 128 bytes on) or weights packed in 64 x 64 blocks
  // (row-major inside, block (row / 64, k / 64) at (row / 64 * K / 64 + k / 64) * 8 KB, next
  // slice 8 KB on: a tile slice reads whole 8 KB blocks).  A chunk past the tile or past N
  // reads from the first byte past the operand: zeros, no memory traffic.
  const int b_oob = (int)(b_bytes > 0x7fffffffLL ? 0x7fffffff : b_bytes);
  const int b_kstride = g.w_packed ? 64 * BK * 2 : BK * 2;
  int b_chunk[CB];
#pragma unroll
  for (int i = 0; i < CB; ++i) {
    const int j = tid + i * NT, row = j >> 3;
    const bool in = j < BN * BK / 8 && n0 + row < g.N;
    if (!g.w_packed)
      b_chunk[i] = in ? b_off + i * b_step : b_oob;
    else
      b_chunk[i] = in ? (int)((((int64_t)((n0 + row) >> 6) * (g.K / 64) + k_base / 64) * 4096 +
                               (row & 63) * 64 + (j & 7) * 8) * 2)
                      : b_oob;
  }

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  u32x4_t ra0[CA], rb0[CB];
  [[maybe_unused]] u32x4_t ra1[CA], rb1[CB];
#define GEMM_FETCH(ra, rb, kt)                                            \
  do {                                                                    \
    buf_load<CA, A_EXACT>(ra, a_rs, a_off + (kt) * BK * 2, a_step, a_last); \
    buf_load_chunks<CB, B_EXACT>(rb, b_rs, b_chunk, (kt) * b_kstride, b_last); \
  } while (0)
  auto stash = [&](int buf, const u32x4_t(&ra)[CA], const u32x4_t(&rb)[CB]) {
#pragma unroll
    for (int i = 0; i < CA; ++i)
      if (A_EXACT || i + 1 < CA || a_last)
        *reinterpret_cast<u32x4_t*>(&As[buf][lds_off + i * LDS_STEP]) = ra[i];
#pragma unroll
    for (int i = 0; i < CB; ++i)
      if (B_EXACT || i + 1 < CB || b_last)
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

  if constexpr (PIPE == 2) {
    bf16x8_t fa0[TM], fb0[TN], fa1[TM], fb1[TN];
    auto stash_a = [&](int buf, const u32x4_t(&ra)[CA]) {
#pragma unroll
      for (int i = 0; i < CA; ++i)
        *reinterpret_cast<u32x4_t*>(&As[buf][lds_off + i * LDS_STEP]) = ra[i];
    };
    auto stash_b = [&](int buf, const u32x4_t(&rb)[CB]) {
#pragma unroll
      for (int i = 0; i < CB; ++i)
        *reinterpret_cast<u32x4_t*>(&Bs[buf][lds_off + i * LDS_STEP]) = rb[i];
    };
    // all chunks of every thread: rows past the tile read real rows or the range-checked
    // zeros past M / N, and are stored to the spare LDS rows
    // a thread's chunk past the tile (CA * NT / 8 > BM) reads from the first byte past the
    // operand: zeros, no memory traffic
    const int a_tail = A_EXACT || a_last ? a_off : (int)(a_bytes > 0x7fffffffLL ? 0x7fffffff : a_bytes);
#define FETCH_ALL(ra, rb, kt)                                                              \
  do {                                                                                     \
    buf_load_tail<CA>(ra, a_rs, a_off + (kt) * BK * 2, a_tail + (kt) * BK * 2, a_step);    \
    buf_load_chunks<CB, true>(rb, b_rs, b_chunk, (kt) * b_kstride, true);                 \
  } while (0)
#define SG(mask, n) __builtin_amdgcn_sched_group_barrier(mask, n, 0)
    // slice KT out of LDS buffer KT & 1; RAN/RBN hold slice KT+1 on entry and receive
    // slice KT+3 (clamped to the last slice)
#define SLICE(KT, RAN, RBN)                                                             \
  do {                                                                                  \
    const int kt_ = (KT), cur = kt_ & 1;                                                \
    load_frags(cur, 16, fa1, fb1);                                                      \
    mfmas(fa0, fb0);                                                                    \
    stash_a(cur ^ 1, RAN);                                                              \
    _Pragma("unroll") for (int q = 0; q < TM * TN; ++q) { SG(0x008, 1); SG(0x100, 1); SG(0x200, 1); } \
    __builtin_amdgcn_sched_barrier(0);                                                  \
    load_frags(cur, 32, fa0, fb0);                                                      \
    mfmas(fa1, fb1);                                                                    \
    stash_b(cur ^ 1, RBN);                                                              \
    _Pragma("unroll") for (int q = 0; q < TM * TN; ++q) { SG(0x008, 1); SG(0x100, 1); SG(0x200, 1); } \
    __builtin_amdgcn_sched_barrier(0);                                                  \
    load_frags(cur, 48, fa1, fb1);                                                      \
    mfmas(fa0, fb0);                                                                    \
    FETCH_ALL(RAN, RBN, kt_ + 3 < nk ? kt_ + 3 : nk - 1);                               \
    _Pragma("unroll") for (int q = 0; q < TM * TN; ++q) { SG(0x008, 1); SG(0x100, 1); SG(0x020, 2); } \
    __builtin_amdgcn_sched_barrier(0);                                                  \
    __syncthreads();                                                                    \
    load_frags(cur ^ 1, 0, fa0, fb0);                                                   \
    mfmas(fa1, fb1);                                                                    \
    _Pragma("unroll") for (int q = 0; q < TM * TN; ++q) { SG(0x008, 1); SG(0x100, 1); }       \
    __builtin_amdgcn_sched_barrier(0);                                                  \
  } while (0)
    FETCH_ALL(ra0, rb0, 0);
    FETCH_ALL(ra1, rb1, nk > 1 ? 1 : 0);
    stash_a(0, ra0);
    stash_b(0, rb0);
    FETCH_ALL(ra0, rb0, nk > 2 ? 2 : nk - 1);
    __syncthreads();
    load_frags(0, 0, fa0, fb0);
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
      SLICE(kt, ra1, rb1);
      SLICE(kt + 1, ra0, rb0);
    }
    if (kt < nk) SLICE(kt, ra1, rb1);
#undef SLICE
#undef SG
#undef FETCH_ALL
  } else if constexpr (PIPE == 1) {
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
  } else {
    // slice kt in LDS, slice kt+1 in registers
    GEMM_FETCH(ra0, rb0, 0);
    stash(0, ra0, rb0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) GEMM_FETCH(ra0, rb0, kt + 1);
      compute(kt & 1);
      if (kt + 1 < nk) stash((kt + 1) & 1, ra0, rb0);
      __syncthreads();
    }
  }
#undef GEMM_FETCH
  // epilogue: acc[i][j][e] is C[row, col] with
  //   row = m0 + wm*TM*32 + i*32 + 8*(e/4) + 4*(lane/32) + e%4,  col = n0 + wn*TN*32 + j*32 + lane%32
  const int col_l = lane & 31, row_q = (lane >> 5) * 4;
  // The SwiGLU, QKV and fp32 epilogues stage each wavefront's finished tile in LDS (the
  // operand buffers are free once every wavefront is past its last slice) and write it back
  // as 16-byte stores: 128 contiguous bytes per row of q, k and the SwiGLU output, per head
  // dimension of the transposed v and per 32 floats of an fp32 row, instead of 2- or 4-byte
  // stores spread over 32 rows.
  constexpr int WR = TM * 32, WC = TN * 32;  // wavefront tile
  if constexpr (EPI == EPI_SWIGLU) {
    constexpr int OC = WC / 2;                // output columns of the tile (gate/up pairs)
    constexpr int SPS = OC + 8;               // staged row pitch, bf16
    static_assert(sizeof(lds) >= (size_t)WAVES_M * WAVES_N * WR * SPS * 2, "stage");
    __syncthreads();                          // every wavefront is done with As / Bs
    uint16_t* scr = lds + wave * WR * SPS;
#pragma unroll
    for (int t = 0; t < TN / 2; ++t)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float gt = acc[i][2 * t][e], up = acc[i][2 * t + 1][e];
          const float sg = gt / (1.0f + __expf(-gt));
          scr[(i * 32 + 8 * (e >> 2) + row_q + (e & 3)) * SPS + t * 32 + col_l] =
              (uint16_t)f32_to_bf16_bits(sg * up);
        }
    __syncthreads();
    uint16_t* C = reinterpret_cast<uint16_t*>(g.C);
    const int pcol0 = n0 + wn * WC;           // first physical column of the wavefront
    const int jcol0 = pcol0 / 2;              // its first output (ffn) column
    const int ncol = min(OC, (g.N - pcol0) / 2);
    constexpr int CPR = OC / 8;               // 16-byte chunks per staged row
    const int64_t row0 = m0 + wm * WR;
    if (ncol > 0) {
#pragma unroll
      for (int k = 0; k < WR * CPR / 64; ++k) {
        const int id = lane + 64 * k, r = id / CPR, cc = (id % CPR) * 8;
        if (row0 + r < g.M && cc < ncol)
          *reinterpret_cast<u32x4_t*>(C + (row0 + r) * g.ldc + jcol0 + cc) =
              *reinterpret_cast<const u32x4_t*>(scr + r * SPS + cc);
      }
    }
  } else if constexpr (EPI == EPI_QKV_ROPE) {
    // q/k columns are pair-interleaved within a head, so the rotate-half partner of
    // column c is column c ^ 1, held by lane ^ 1 for the same rows.  A wavefront's WC
    // columns lie in one head of one section (q, k or v): section widths are multiples of
    // 64.  q and k are staged row-major and leave as rows of the head layout; v is staged
    // transposed and leaves as runs of 8 positions of the transposed layout.
    const QkvOut& o = g.qkv;
    const int hd = o.head_dim, half = hd / 2;
    const int hq = o.n_heads * hd, hkv = o.n_kv_heads * hd;
    const int c0 = n0 + wn * WC;
    const int sec = c0 < hq ? 0 : (c0 < hq + hkv ? 1 : 2);
    const int cc0 = c0 - (sec == 0 ? 0 : (sec == 1 ? hq : hq + hkv));
    const int head = cc0 / hd, pd0 = cc0 % hd;
    constexpr int SPS = WC + 8, SPV = WR + 8;  // staged pitches, bf16
    static_assert(sizeof(lds) >= (size_t)WAVES_M * WAVES_N * WR * SPS * 2 &&
                  sizeof(lds) >= (size_t)WAVES_M * WAVES_N * WC * SPV * 2, "stage");
    __syncthreads();                           // every wavefront is done with As / Bs
    uint16_t* scr = lds + wave * (WR * SPS > WC * SPV ? WR * SPS : WC * SPV);
    const int64_t row0 = m0 + wm * WR;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = c0 + j * 32 + col_l;
      const float bias = (col < g.N && g.bias) ? g.bias[col] : 0.f;
      const int ii = (pd0 + j * 32 + col_l) >> 1;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {  // rows 8 e4 + .. of e4 = 2 hf, 2 hf + 1
          float x[2][4], partner[2][4];
#pragma unroll
          for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              x[u][t] = acc[i][j][(2 * hf + u) * 4 + t] + bias;
              partner[u][t] = __shfl_xor(x[u][t], 1, 64);
            }
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int rl = i * 32 + row_q + 16 * hf + 8 * u;  // staged row of element t = 0
            if (sec < 2) {
              // the cos/sin loads of these 4 elements are issued before the LDS writes
              float cs[4], sn[4];
              int pos = (int)((row0 + rl) % o.L);
#pragma unroll
              for (int t = 0; t < 4; ++t) {
                cs[t] = o.cos_t[pos * half + ii];
                sn[t] = o.sin_t[pos * half + ii];
                if (++pos == o.L) pos = 0;
              }
#pragma unroll
              for (int t = 0; t < 4; ++t) {
                const float r = (col_l & 1) ? x[u][t] * cs[t] + partner[u][t] * sn[t]
                                            : x[u][t] * cs[t] - partner[u][t] * sn[t];
                scr[(rl + t) * SPS + j * 32 + col_l] = (uint16_t)f32_to_bf16_bits(r);
              }
            } else {
              u32x2_t v2;
              v2.x = pack_bf16x2(x[u][0], x[u][1]);
              v2.y = pack_bf16x2(x[u][2], x[u][3]);
              *reinterpret_cast<u32x2_t*>(scr + (j * 32 + col_l) * SPV + rl) = v2;
            }
          }
        }
    }
    __syncthreads();
    if (c0 < g.N) {
      if (sec < 2) {
        constexpr int CPR = WC / 8;            // 16-byte chunks per staged row
        uint16_t* base = sec == 0 ? o.q : o.k;
        const int nh = sec == 0 ? o.n_heads : o.n_kv_heads;
#pragma unroll
        for (int k = 0; k < WR * CPR / 64; ++k) {
          const int id = lane + 64 * k, r = id / CPR, cc = (id % CPR) * 8;
          const int64_t m = row0 + r;
          if (m < g.M) {
            const int b = (int)(m / o.L), pos = (int)(m - (int64_t)b * o.L);
            *reinterpret_cast<u32x4_t*>(base + ((int64_t)(b * nh + head) * o.Ls + pos) * hd +
                                        pd0 + cc) =
                *reinterpret_cast<const u32x4_t*>(scr + r * SPS + cc);
          }
        }
      } else {
        constexpr int CPC = WR / 8;            // runs of 8 positions per head dimension
#pragma unroll
        for (int k = 0; k < WC * CPC / 64; ++k) {
          const int id = lane + 64 * k, dcol = id / CPC, rr = (id % CPC) * 8;
          const int64_t m = row0 + rr;
          const int b = (int)(m / o.L), pos = (int)(m - (int64_t)b * o.L);
          uint16_t* dst = o.vt + ((int64_t)(b * o.n_kv_heads + head) * hd + pd0 + dcol) * o.Ls;
          if (m + 7 < g.M && pos + 7 < o.L && (pos & 7) == 0) {
            *reinterpret_cast<u32x4_t*>(dst + pos) =
                *reinterpret_cast<const u32x4_t*>(scr + dcol * SPV + rr);
          } else {
            int bb = b, pp = pos;
            for (int t = 0; t < 8 && m + t < g.M; ++t) {
              o.vt[((int64_t)(bb * o.n_kv_heads + head) * hd + pd0 + dcol) * o.Ls + pp] =
                  scr[dcol * SPV + rr + t];
              if (++pp == o.L) { pp = 0; ++bb; }
            }
          }
        }
      }
    }
  } else if constexpr (EPI == EPI_TOP1) {
    // Row statistics of Eq. (1) over this wavefront's TN x 32 columns.  Each 32 x 32 block
    // passes through a per-wavefront LDS scratch as the rounded logits EPI_BF16 would write;
    // lane l reduces row l % 32 over the block's columns 16 (l / 32) .. + 15, the two lanes
    // of a row are merged (lower columns first), and the blocks of a block row are folded in
    // column order.
    constexpr int SP = 34;  // scratch row pitch, bf16
    static_assert(sizeof(lds) >= (size_t)WAVES_M * WAVES_N * 32 * SP * 2, "TOP1 scratch");
    __syncthreads();  // every wavefront is done reading the operand tiles
    uint16_t* scr = lds + wave * 32 * SP;
    const int rr = lane & 31, half = lane >> 5;
    TopState rs[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) rs[i] = TopState{-INFINITY, 0.f, INT_MAX};
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int e = 0; e < 16; ++e)
          scr[(8 * (e >> 2) + row_q + (e & 3)) * SP + col_l] =
              (uint16_t)f32_to_bf16_bits(acc[i][j][e] * g.scale);
        __syncthreads();
        const int c0 = n0 + wn * TN * 32 + j * 32 + half * 16;
        float v[16];
        TopState t{-INFINITY, 0.f, INT_MAX};
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          float x = bf16_bits_to_f32(scr[rr * SP + half * 16 + c]);
          if (c0 + c >= g.N || c0 + c == g.mask_id) x = -INFINITY;
          v[c] = x;
          if (x > t.m) { t.m = x; t.arg = c0 + c; }
        }
        if (t.m != -INFINITY) {
          const float ml = t.m * LOG2E;
#pragma unroll
          for (int c = 0; c < 16; ++c) t.s += fast_exp2(fmaf(v[c], LOG2E, -ml));
        }
        const TopState u{__shfl_xor(t.m, 32, 64), __shfl_xor(t.s, 32, 64), __shfl_xor(t.arg, 32, 64)};
        rs[i] = merge(rs[i], half == 0 ? merge(t, u) : merge(u, t));
        __syncthreads();  // the scratch is rewritten by the next block
      }
    const int part = tile_n * WAVES_N + wn;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int row = m0 + wm * TM * 32 + i * 32 + rr;
      if (half == 0 && row < g.M) {
        const int64_t o = (int64_t)row * g.n_parts + part;
        g.part_m[o] = rs[i].m;
        g.part_s[o] = rs[i].s;
        g.part_arg[o] = rs[i].arg;
      }
    }
  } else if constexpr (EPI == EPI_ADD_F32 || EPI == EPI_PART_F32) {
    // fp32 outputs (residual update, split-K partials): each wavefront stages one 32-row
    // block of its tile at a time in LDS (a whole fp32 tile per wavefront would not fit) and
    // writes rows of WC floats as 16-byte stores, a read-modify-write for the residual update
    constexpr int SPF = WC + 4;                // staged row pitch, fp32
    constexpr int CPR = WC / 4;                // 16-byte chunks per staged row
    static_assert(sizeof(lds) >= (size_t)WAVES_M * WAVES_N * 32 * SPF * 4, "stage");
    float* scr = reinterpret_cast<float*>(lds) + wave * 32 * SPF;
    float* C = reinterpret_cast<float*>(g.C) +
               (EPI == EPI_PART_F32 ? (int64_t)split * g.M * g.ldc : (int64_t)0);
    const int c0 = n0 + wn * WC;
    const int ncol = min(WC, g.N - c0);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      __syncthreads();  // the operand buffers (i = 0) or the previous block are done with
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          scr[(8 * (e >> 2) + row_q + (e & 3)) * SPF + j * 32 + col_l] = acc[i][j][e];
      __syncthreads();
      const int64_t row0 = m0 + wm * WR + i * 32;
      if (ncol > 0) {
#pragma unroll
        for (int k = 0; k < 32 * CPR / 64; ++k) {
          const int id = lane + 64 * k, r = id / CPR, cc = (id % CPR) * 4;
          if (row0 + r >= g.M || cc >= ncol) continue;
          float* dst = C + (row0 + r) * g.ldc + c0 + cc;
          const float* src = scr + r * SPF + cc;
          if (cc + 4 <= ncol) {
            float4 v = *reinterpret_cast<const float4*>(src);
            if constexpr (EPI == EPI_ADD_F32) {
              const float4 h = *reinterpret_cast<const float4*>(dst);
              v.x = h.x + v.x;
              v.y = h.y + v.y;
              v.z = h.z + v.z;
              v.w = h.w + v.w;
            }
            *reinterpret_cast<float4*>(dst) = v;
          } else {
            for (int t = 0; t < ncol - cc; ++t) dst[t] = EPI == EPI_ADD_F32 ? dst[t] + src[t] : src[t];
          }
        }
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * TN * 32 + j * 32 + col_l;
      if (col >= g.N) continue;
      const float bias = g.bias ? g.bias[col] : 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * TM * 32 + i * 32 + 8 * (e >> 2) + row_q + (e & 3);
          if (row >= g.M) continue;
          uint16_t* C = reinterpret_cast<uint16_t*>(g.C);
          C[(int64_t)row * g.ldc + col] =
              (uint16_t)f32_to_bf16_bits((acc[i][j][e] + bias) * g.scale);
        }
    }
  }
}

// ---- tile configurations ---------------------------------------------------------------
// LDS read throughput per CU grows with the number of resident waves (one wave per SIMD
// cannot keep enough reads in flight to feed the MFMA pipe), so the large-tile configs
// run 2-4 waves per SIMD.
// cfg 0: 256 x 256 tile, 16 waves (4 x 4), wave tile 64 x 64, PIPE 0
// cfg 1:  32 x 128 tile, 4 waves (1 x 4) (2 waves for SwiGLU), for M <= 64 (LM head rows)
// cfg 2: 256 x 128 tile,  8 waves (4 x 2), wave tile 64 x 64, PIPE 2
// cfg 3: 256 x 192 tile, 12 waves (4 x 3), wave tile 64 x 64, PIPE 2
// cfg 4: 128 x 192 tile, 12 waves (4 x 3), wave tile 32 x 64, PIPE 2: twice the tiles of
//        cfg 3, so an output of 512 rows x 12288 columns fills 256 CUs without splitting K.
//        Twelve waves load the four SIMDs evenly (three each); as 6 waves of 64 x 64 (two
//        SIMDs with two waves, two with one) the QKV projection at 512 rows ran 1.2 %
//        slower per pass, although a 32 x 64 wave tile reads 1.5 x the LDS bytes per MFMA
struct CfgShape { int bm, bn; };
static CfgShape cfg_shape(int cfg) {
  switch (cfg) {
    case 0: return {256, 256};
    case 1: return {32, 128};
    case 3: return {256, 192};
    case 4: return {128, 192};
    default: return {256, 128};
  }
}

int gemm_num_cfgs() { return 5; }

// wavefront columns per tile and their width (TN x 32) of each config
int gemm_top1_parts(const GemmPlan& p, int N) {
  const CfgShape sh = cfg_shape(p.cfg);
  const int waves_n = p.cfg == 0 ? 4 : (p.cfg == 1 ? 4 : (p.cfg == 3 || p.cfg == 4 ? 3 : 2));
  return (N + sh.bn - 1) / sh.bn * waves_n;
}

// Relative main-loop efficiency of the large-tile configs (16, 12, 8 and 12 waves per
// workgroup), measured on the pass's shapes (cfg 4: 64.4 us for the whole-K QKV projection
// with its bias + RoPE epilogue at 512 x 12288 x 4096, as 6 waves; the 12-wave layout is a
// few us faster there, and keeping the 6-wave figure leaves every plan as it was).
static double cfg_eff(int cfg) {
  return cfg == 0 ? 1.0 : (cfg == 3 ? 1.03 : (cfg == 4 ? 0.72 : 0.88));
}

GemmPlan gemm_plan_cfg(int M, int N, int K, int cfg, int splits) {
  GemmPlan p{};
  p.cfg = cfg;
  const CfgShape sh = cfg_shape(cfg);
  p.tiles = ((M + sh.bm - 1) / sh.bm) * ((N + sh.bn - 1) / sh.bn);
  p.splits = splits;
  p.ws_floats = splits > 1 ? (size_t)splits * M * N : 0;
  return p;
}

// Whole-K tiles: minimise rounds-of-tiles x tile area / efficiency, which picks the fastest
// measured config at every shape of the pass (e.g. 256 x 192 for the 512 x 24576 gate/up,
// 256 x 128 for 512 x 12288).
GemmPlan gemm_plan(int M, int N, int K, int num_cus) {
  if (M <= 64) return gemm_plan_cfg(M, N, K, 1, 1);
  const int cfgs[4] = {0, 3, 2, 4};
  int best = 0;
  double best_cost = 0;
  for (int c = 0; c < 4; ++c) {
    const CfgShape sh = cfg_shape(cfgs[c]);
    const int tiles = ((M + sh.bm - 1) / sh.bm) * ((N + sh.bn - 1) / sh.bn);
    const int rounds = (tiles + num_cus - 1) / num_cus;
    const double cost = (double)rounds * sh.bm * sh.bn / cfg_eff(cfgs[c]);
    if (c == 0 || cost < best_cost) { best = cfgs[c]; best_cost = cost; }
  }
  return gemm_plan_cfg(M, N, K, best, 1);
}

// Tiles that may split K (outputs whose consumer folds partials in): estimated time =
// rounds x per-tile main loop (2.18 MMAC per microsecond per CU at efficiency 1) + partial
// traffic (written here, read back downstream: ~0.46 us per MiB, the measured cost of the
// QKV split-K 2 partials and their finish kernel), over configs {0, 2, 3, 4} and
// 1, 2, 4 or 8 splits with >= 8 K-slices each (only `splits` when it is > 0).  Splits never
// exceed the workspace bound.
GemmPlan gemm_plan_split(int M, int N, int K, int num_cus, int splits) {
  if (M <= 64 && splits <= 1) return gemm_plan_cfg(M, N, K, 1, 1);
  const int nk = K / BK;
  const int cfgs[4] = {0, 3, 2, 4};
  GemmPlan best{};
  double best_us = 0;
  bool have = false;
  for (int c = 0; c < 4; ++c) {
    const CfgShape sh = cfg_shape(cfgs[c]);
    const int tiles = ((M + sh.bm - 1) / sh.bm) * ((N + sh.bn - 1) / sh.bn);
    for (int sp = 1; sp <= 8; sp *= 2) {
      if (splits > 0 && sp != splits) continue;
      if (sp > 1 && (nk % sp != 0 || nk / sp < 8 ||
                     (size_t)sp * M * N > gemm_ws_floats_bound(num_cus)))
        continue;
      const int rounds = (tiles * sp + num_cus - 1) / num_cus;
      double us = (double)rounds * sh.bm * sh.bn * ((double)K / sp) / cfg_eff(cfgs[c]) / 2.18e6;
      if (sp > 1) us += 0.46 * (double)sp * M * N * 4.0 / (1 << 20);
      if (!have || us < best_us) { best = gemm_plan_cfg(M, N, K, cfgs[c], sp); best_us = us; have = true; }
    }
  }
  return best;
}

// With timing events, the dispatch itself stamps them with the kernel's start and end
// (hipExtLaunchKernel), so no marker packet sits between the events and the kernel.
template <int WAVES_M, int WAVES_N, int TM, int TN, int EPI, int PIPE>
static hipError_t run(const GemmArgs& a, int grid, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (e0 || e1)
    hipExtLaunchKernelGGL((k_gemm<WAVES_M, WAVES_N, TM, TN, EPI, PIPE>), dim3(grid),
                          dim3(WAVES_M * WAVES_N * 64), 0, s, e0, e1, 0, a);
  else
    hipLaunchKernelGGL((k_gemm<WAVES_M, WAVES_N, TM, TN, EPI, PIPE>), dim3(grid),
                       dim3(WAVES_M * WAVES_N * 64), 0, s, a);
  return hipGetLastError();
}

template <int EPI>
static hipError_t run_cfg(int cfg, const GemmArgs& a, int grid, hipStream_t s, hipEvent_t e0,
                          hipEvent_t e1) {
  switch (cfg) {
    case 0: return run<4, 4, 2, 2, EPI, 0>(a, grid, s, e0, e1);
    case 1:
      if constexpr (EPI == EPI_SWIGLU) return run<1, 2, 1, 2, EPI, 1>(a, grid, s, e0, e1);
      else return run<1, 4, 1, 1, EPI, 1>(a, grid, s, e0, e1);
    case 3: return run<4, 3, 2, 2, EPI, 2>(a, grid, s, e0, e1);
    case 4: return run<4, 3, 1, 2, EPI, 2>(a, grid, s, e0, e1);
    default: return run<4, 2, 2, 2, EPI, 2>(a, grid, s, e0, e1);
  }
}

hipError_t launch_gemm(int epi, const GemmArgs& in, const GemmPlan& p, hipStream_t s,
                       hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (in.M == 0 || in.N == 0) return hipSuccess;
  if (p.splits < 1 || in.K % (BK * p.splits) != 0) return hipErrorInvalidValue;
  if (p.splits > 1 && epi != EPI_PART_F32) return hipErrorInvalidValue;
  GemmArgs a = in;
  a.splits = p.splits;
  const int grid = p.tiles * p.splits;
  switch (epi) {
    case EPI_BF16: return run_cfg<EPI_BF16>(p.cfg, a, grid, s, ev_start, ev_stop);
    case EPI_ADD_F32: return run_cfg<EPI_ADD_F32>(p.cfg, a, grid, s, ev_start, ev_stop);
    case EPI_SWIGLU: return run_cfg<EPI_SWIGLU>(p.cfg, a, grid, s, ev_start, ev_stop);
    case EPI_QKV_ROPE: return run_cfg<EPI_QKV_ROPE>(p.cfg, a, grid, s, ev_start, ev_stop);
    case EPI_PART_F32: return run_cfg<EPI_PART_F32>(p.cfg, a, grid, s, ev_start, ev_stop);
    case EPI_TOP1:
      if (a.n_parts != gemm_top1_parts(p, a.N) || !a.part_m || !a.part_s || !a.part_arg)
        return hipErrorInvalidValue;
      return run_cfg<EPI_TOP1>(p.cfg, a, grid, s, ev_start, ev_stop);
  }
  return hipErrorInvalidValue;
}

}  // namespace cora
