// LM head for few rows (M <= 64): logits = bf16((A . W^T) * scale) with A [M, K] the
// normalised rows and W [N, K] the vocab projection, and the same pass fused with the
// row statistics of Eq. (1).
//
// At a 32-row block the product is a pure weight stream (1 GB at LLaDA-8B size, 32 flops
// per weight byte), so the kernel is built for HBM, not for the matrix cores.  HBM delivers
// ~6.8 TB/s to loads that cover 1 KB of contiguous memory per instruction, but only ~5.1
// TB/s when an instruction covers 128 bytes of each of 8 rows 8 KB apart (the tile loads of
// a row-major GEMM), so the weights are read from a packed copy made once at model
// creation, laid out in the order this kernel consumes it:
//   * wavefront G owns vocab rows 32 G .. 32 G + 31 (two 16-row MFMA blocks) over all of K;
//     its 32 x K weights are one contiguous region of 1 KB blocks, block (stage st, block
//     wb, step s) = rows 32 G + 16 wb + (0..15), k = 64 st + 32 s + (0..31), stored as the
//     v_mfma_f32_16x16x32_bf16 operand: lane l = r + 16 q holds row r, k 8 q .. 8 q + 7;
//   * one 16-byte load per lane reads one block, so a stage (4 blocks) is 4 KB of
//     contiguous memory, and D stages are in flight in a register ring;
//   * the activations of a stage (M x 64) are loaded once per workgroup (one 16-byte chunk
//     per thread and 32 rows), stored to a double-buffered LDS tile and read back as MFMA
//     fragments by all four wavefronts: one barrier per stage;
//   * no LDS holds weights (~9 KB per workgroup), so all 988 workgroups of a 126464-entry
//     vocab are resident at once.
// Stages past K read out of range (zeros, no memory traffic), so the loop body has no
// branches and the ring index stays compile-time.
//
// TOP1 mode writes no logits: the rounded logits of a workgroup's 128 vocab entries are
// reduced per row to (max, lowest arg max, sum exp(l - max)) with the mask id left out, and
// k_top1_merge folds a row's partials in vocab order into the top-1 token and confidence
// c = 1 / sum_v exp(l_v - l_max).  Both modes round the same accumulators the same way, so
// the fused statistics are those of the logits the plain mode writes.
#include <limits.h>

#include "common.hpp"
#include "internal.hpp"

namespace cora {

constexpr int LMH_WAVES = 4, LMH_ROWS_PER_WAVE = 32;
constexpr int LMH_COLS = LMH_WAVES * LMH_ROWS_PER_WAVE;  // vocab entries per workgroup
constexpr int LMH_STAGE_K = 64;
constexpr int LMH_LDA = LMH_STAGE_K + 8;                 // padded LDS row (bf16 elements)
// cache policy of the weight loads: nontemporal (each weight byte is read once per call)
#ifndef LMH_W_POLICY
#define LMH_W_POLICY 2
#endif

int lm_head_parts(int N) { return (N + LMH_COLS - 1) / LMH_COLS; }
__host__ __device__ inline int64_t packed_elems(int N, int K) { return (int64_t)((N + 31) / 32) * 32 * K; }
size_t lm_head_packed_elems(int N, int K) { return (size_t)packed_elems(N, K); }

// packed[G][st][wb][s][l][j] = W[32 G + 16 wb + l % 16][64 st + 32 s + 8 (l / 16) + j] (zero
// past N): thread = one 16-byte chunk of the packed copy
__global__ __launch_bounds__(256) void k_pack_lm_head(const uint16_t* __restrict__ W,
                                                      uint16_t* __restrict__ P, int N, int K) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_g = (int64_t)K * 4;  // chunks per 32-row group
  if (c >= (int64_t)((N + 31) / 32) * per_g) return;
  const int G = (int)(c / per_g);
  const int rem = (int)(c - G * per_g);
  const int blk = rem >> 6, l = rem & 63;
  const int st = blk >> 2, wb = (blk >> 1) & 1, s = blk & 1;
  const int row = 32 * G + 16 * wb + (l & 15), k = 64 * st + 32 * s + 8 * (l >> 4);
  u32x4_t v = {0u, 0u, 0u, 0u};
  if (row < N) v = *reinterpret_cast<const u32x4_t*>(W + (int64_t)row * K + k);
  *reinterpret_cast<u32x4_t*>(P + c * 8) = v;
}

hipError_t launch_pack_lm_head(const uint16_t* W, uint16_t* packed, int N, int K,
                               hipStream_t s) {
  if (N <= 0 || K % LMH_STAGE_K != 0) return hipErrorInvalidValue;
  const int64_t chunks = packed_elems(N, K) / 8;
  hipLaunchKernelGGL(k_pack_lm_head, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, s, W,
                     packed, N, K);
  return hipGetLastError();
}

// MB = 16-row blocks of activation rows (M <= 16 * MB), D = stages in the register ring
template <int MB, int D, bool TOP1>
__global__ __launch_bounds__(256) void k_lm_head(LmHeadArgs a) {
  constexpr int AR = 16 * MB;                  // activation rows held per stage
  constexpr int ACH = AR * LMH_STAGE_K / 8 / 256;  // 16-byte A chunks per thread per stage
  static_assert(ACH >= 1 && ACH * 256 * 8 == AR * LMH_STAGE_K, "A stage must split evenly");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][AR * LMH_LDA];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, q = lane >> 4;
  const int n_wave = blockIdx.x * LMH_COLS + wave * LMH_ROWS_PER_WAVE;

  // buffer resources: activation rows past M read as zero; the packed weights are zero
  // past N already
  const int64_t w_bytes = packed_elems(a.N, a.K) * 2;
  const int64_t a_bytes = (int64_t)a.M * a.lda * 2;
  const __amdgpu_buffer_rsrc_t w_rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)a.Wp, (short)0, (int)(w_bytes > 0x7fffffffLL ? 0x7fffffff : w_bytes), 0x00020000);
  const __amdgpu_buffer_rsrc_t a_rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)a.A, (short)0, (int)(a_bytes > 0x7fffffffLL ? 0x7fffffff : a_bytes), 0x00020000);
  constexpr int OOB = 0x7fffffff;  // an offset past every buffer: zeros, no traffic

  // weights: this lane's 16 bytes of block (st, wb, s) of group G = n_wave / 32 (a group
  // past the packed copy, in the last workgroup, reads zeros)
  const int64_t g_bytes = (int64_t)(n_wave / 32) * 32 * a.K * 2;
  const bool w_in = g_bytes < w_bytes;
  const int w_base = w_in ? (int)g_bytes + lane * 16 : 0;
  // activations: chunk c of this thread is row (tid / 8) + 32 c, k = 8 (tid % 8)
  const int a_r = tid >> 3, a_k = (tid & 7) * 8;
  int a_off[ACH];
#pragma unroll
  for (int c = 0; c < ACH; ++c) {
    const int row = a_r + 32 * c;
    a_off[c] = row < a.M ? (int)(((int64_t)row * a.lda + a_k) * 2) : OOB;
  }
  const int nst = a.K / LMH_STAGE_K;

  u32x4_t wr[D][2][2];
  u32x4_t ar[D][ACH];
  auto issue = [&](int st, u32x4_t (&w)[2][2], u32x4_t (&x)[ACH]) {
    const bool in = st < nst;
    const int kb = st * LMH_STAGE_K * 2;  // activation bytes
#pragma unroll
    for (int c = 0; c < ACH; ++c)
      x[c] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                             a_rs, in ? a_off[c] + kb : OOB, 0, 0));
#pragma unroll
    for (int wb = 0; wb < 2; ++wb)
#pragma unroll
      for (int s = 0; s < 2; ++s)
        w[wb][s] = __builtin_bit_cast(
            u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(w_rs, in && w_in ? w_base + st * 4096 : OOB,
                                                           (2 * wb + s) * 1024, LMH_W_POLICY));
  };

  f32x4_t acc[2][MB];
#pragma unroll
  for (int wb = 0; wb < 2; ++wb)
#pragma unroll
    for (int ab = 0; ab < MB; ++ab) acc[wb][ab] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int u = 0; u + 1 < D; ++u) {
    issue(u, wr[u], ar[u]);
    __builtin_amdgcn_sched_barrier(0);
  }

  const int a_st = a_r * LMH_LDA + a_k;
  const int n_iter = (nst + D - 1) / D * D;
  for (int st0 = 0; st0 < n_iter; st0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int st = st0 + u;
      // scheduling barriers keep every stage's loads in issue order, so the wait for
      // stage st leaves the D - 1 younger stages in flight
      issue(st + D - 1, wr[(u + D - 1) % D], ar[(u + D - 1) % D]);
      __builtin_amdgcn_sched_barrier(0);
      uint16_t* buf = As[u & 1];  // D is even: stage parity == u parity
#pragma unroll
      for (int c = 0; c < ACH; ++c)
        *reinterpret_cast<u32x4_t*>(&buf[a_st + 32 * c * LMH_LDA]) = ar[u][c];
      __syncthreads();
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        bf16x8_t fa[MB];
#pragma unroll
        for (int ab = 0; ab < MB; ++ab)
          fa[ab] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(
              &buf[(ab * 16 + r16) * LMH_LDA + 32 * s + 8 * q]));
#pragma unroll
        for (int wb = 0; wb < 2; ++wb)
#pragma unroll
          for (int ab = 0; ab < MB; ++ab)
            acc[wb][ab] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wr[u][wb][s]), fa[ab],
                                                                 acc[wb][ab], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // acc[wb][ab][e] = logits of row ab * 16 + r16 at vocab n_wave + 16 wb + 4 q + e
  if constexpr (!TOP1) {
#pragma unroll
    for (int ab = 0; ab < MB; ++ab) {
      const int row = ab * 16 + r16;
      if (row >= a.M) continue;
      uint16_t* dst = a.logits + (int64_t)row * a.ldc;
#pragma unroll
      for (int wb = 0; wb < 2; ++wb) {
        const int v = n_wave + 16 * wb + 4 * q;
        const f32x4_t x = acc[wb][ab];
        if (v + 3 < a.N && (a.ldc & 3) == 0) {
          u32x2_t p;
          p.x = pack_bf16x2(x[0] * a.scale, x[1] * a.scale);
          p.y = pack_bf16x2(x[2] * a.scale, x[3] * a.scale);
          *reinterpret_cast<u32x2_t*>(dst + v) = p;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (v + e < a.N) dst[v + e] = (uint16_t)f32_to_bf16_bits(x[e] * a.scale);
        }
      }
    }
  } else {
    // per row: this lane's 8 entries in increasing vocab order, then the 4 lanes of the row
    // (xor 16, 32), then the 4 wavefronts through LDS in vocab order
    __shared__ float sm_m[LMH_WAVES][AR], sm_s[LMH_WAVES][AR];
    __shared__ int sm_a[LMH_WAVES][AR];
#pragma unroll
    for (int ab = 0; ab < MB; ++ab) {
      float v8[8];
      float m = -INFINITY;
      int arg = INT_MAX;
#pragma unroll
      for (int wb = 0; wb < 2; ++wb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int v = n_wave + 16 * wb + 4 * q + e;
          float x = bf16_bits_to_f32(f32_to_bf16_bits(acc[wb][ab][e] * a.scale));
          if (v >= a.N || v == a.mask_id) x = -INFINITY;
          v8[4 * wb + e] = x;
          if (x > m) { m = x; arg = v; }
        }
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float om = __shfl_xor(m, o, 64);
        const int oa = __shfl_xor(arg, o, 64);
        arg = om > m ? oa : (m > om ? arg : min(arg, oa));
        m = fmaxf(m, om);
      }
      float s = 0.f;
      if (m != -INFINITY) {
        const float ml = m * LOG2E;
#pragma unroll
        for (int i = 0; i < 8; ++i) s += fast_exp2(fmaf(v8[i], LOG2E, -ml));
      }
      s += __shfl_xor(s, 16, 64);
      s += __shfl_xor(s, 32, 64);
      if (q == 0) {
        sm_m[wave][ab * 16 + r16] = m;
        sm_s[wave][ab * 16 + r16] = s;
        sm_a[wave][ab * 16 + r16] = arg;
      }
    }
    __syncthreads();
    if (tid < AR && tid < a.M) {
      TopState t{sm_m[0][tid], sm_s[0][tid], sm_a[0][tid]};
#pragma unroll
      for (int w = 1; w < LMH_WAVES; ++w) t = merge(t, TopState{sm_m[w][tid], sm_s[w][tid], sm_a[w][tid]});
      const int64_t o = (int64_t)tid * a.n_parts + blockIdx.x;
      a.part_m[o] = t.m;
      a.part_s[o] = t.s;
      a.part_arg[o] = t.arg;
    }
  }
}

// One workgroup per row: fold the row's partials in vocab order into top-1 and confidence
// (written like the logits-row reduction: row r of batch row b goes to b * out_ld + out_off + r).
__global__ __launch_bounds__(256) void k_top1_merge(const float* __restrict__ pm,
                                                    const float* __restrict__ ps,
                                                    const int* __restrict__ pa, int n_parts,
                                                    int n_rows, int out_ld, int out_off,
                                                    int32_t* __restrict__ top1,
                                                    float* __restrict__ conf) {
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t base = (int64_t)row * n_parts;
  // thread tid folds a contiguous run of partials, so the fold order is vocab order
  const int per = (n_parts + 255) / 256;
  const int p0 = tid * per, p1 = min(p0 + per, n_parts);
  TopState t{-INFINITY, 0.f, INT_MAX};
  for (int p = p0; p < p1; ++p) t = merge(t, TopState{pm[base + p], ps[base + p], pa[base + p]});
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    TopState u;
    u.m = __shfl_xor(t.m, o, 64);
    u.s = __shfl_xor(t.s, o, 64);
    u.arg = __shfl_xor(t.arg, o, 64);
    // the lower lane's runs come first: keep (lower, upper) operand order on both sides
    t = (lane & o) ? merge(u, t) : merge(t, u);
  }
  __shared__ float sm_m[4], sm_s[4];
  __shared__ int sm_a[4];
  if (lane == 0) { sm_m[wave] = t.m; sm_s[wave] = t.s; sm_a[wave] = t.arg; }
  __syncthreads();
  if (tid == 0) {
    TopState r{sm_m[0], sm_s[0], sm_a[0]};
    for (int w = 1; w < 4; ++w) r = merge(r, TopState{sm_m[w], sm_s[w], sm_a[w]});
    const int b = row / n_rows;
    const int64_t o = (int64_t)b * out_ld + out_off + (row - b * n_rows);
    top1[o] = r.arg;
    conf[o] = 1.0f / r.s;
  }
}

bool lm_head_supported(int M, int N, int K, int64_t lda) {
  return M >= 1 && M <= LM_HEAD_FUSED_MAX_ROWS && N >= 1 && K % LMH_STAGE_K == 0 &&
         packed_elems(N, K) * 2 <= 0x7fffffffLL &&
         (int64_t)M * lda * 2 <= 0x7fffffffLL;
}

hipError_t launch_lm_head(const LmHeadArgs& in, bool top1, hipStream_t s) {
  if (!lm_head_supported(in.M, in.N, in.K, in.lda)) return hipErrorInvalidValue;
  LmHeadArgs a = in;
  a.n_parts = lm_head_parts(a.N);
  const dim3 grid(a.n_parts), block(256);
#define LMH(MB_, T_) hipLaunchKernelGGL((k_lm_head<MB_, 4, T_>), grid, block, 0, s, a)
  if (a.M <= 32) {
    if (top1) LMH(2, true);
    else LMH(2, false);
  } else {
    if (top1) LMH(4, true);
    else LMH(4, false);
  }
#undef LMH
  return hipGetLastError();
}

hipError_t launch_top1_merge_parts(const float* pm, const float* ps, const int* pa, int n_parts,
                                   int M, int n_rows, int out_ld, int out_off, int32_t* top1,
                                   float* conf, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (n_parts <= 0 || n_rows <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_top1_merge, dim3(M), dim3(256), 0, s, pm, ps, pa, n_parts, n_rows, out_ld,
                     out_off, top1, conf);
  return hipGetLastError();
}

hipError_t launch_top1_merge(const LmHeadArgs& a, int n_rows, int out_ld, int out_off,
                             int32_t* top1, float* conf, hipStream_t s) {
  return launch_top1_merge_parts(a.part_m, a.part_s, a.part_arg, lm_head_parts(a.N), a.M, n_rows,
                                 out_ld, out_off, top1, conf, s);
}

}  // namespace cora
