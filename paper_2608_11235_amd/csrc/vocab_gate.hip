// Fused vocab reduction + decision rules (one launch per denoising step).
//
// Phase 1, one workgroup per logits row: a single coalesced pass over the bf16 row
// (16-byte loads) keeps a running (max, first argmax, sum of exp(l - max)) per thread,
// merged across the wavefront with xor shuffles and across the 4 wavefronts through
// LDS in a fixed order, so results are bitwise reproducible.  The row's top-1 token
// is the lowest id among equal maxima, the mask id is skipped, and the confidence
// is c = max softmax = 1 / sum_v exp(l_v - l_max) (Eq. 1).
//
// Phase 2, the last workgroup of each batch row to finish (a per-row ticket taken after
// its agent-coherent result stores completed) applies, on that row's active block:
//   block step 0 -> previous top-1 and counters reset (persistence is per block);
//   Eq. (2) counter update on unresolved positions;
//   transfer rule: the k highest-confidence unresolved positions (ties -> lower position);
//   Eq. (3) gate on the other unresolved positions (c >= delta_p and m >= m_req);
//   Eq. (4) commit of both sets; block done once no unresolved position is left,
//   then the row moves to its next block.
// The ticket counter is reset to zero by the workgroup that used it.
#include <limits.h>

#include "common.hpp"
#include "internal.hpp"

namespace cora {

struct TopState {
  float m, s;
  int arg;
};

__device__ __forceinline__ TopState merge(TopState x, TopState y) {
  TopState r;
  r.m = fmaxf(x.m, y.m);
  const float sx = x.m == -INFINITY ? 0.f : x.s * exp2f((x.m - r.m) * 1.4426950408889634f);
  const float sy = y.m == -INFINITY ? 0.f : y.s * exp2f((y.m - r.m) * 1.4426950408889634f);
  r.s = sx + sy;
  r.arg = x.m > y.m ? x.arg : (y.m > x.m ? y.arg : min(x.arg, y.arg));
  return r;
}

__device__ __forceinline__ void consume8(TopState& t, const float (&v)[8], int idx0) {
  float cm = v[0];
  int ca = 0;
#pragma unroll
  for (int j = 1; j < 8; ++j)
    if (v[j] > cm) { cm = v[j]; ca = j; }
  if (cm > t.m) {
    t.s = t.m == -INFINITY ? 0.f : t.s * exp2f((t.m - cm) * 1.4426950408889634f);
    t.m = cm;
    t.arg = idx0 + ca;
  }
  if (t.m == -INFINITY) return;
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) acc += exp2f((v[j] - t.m) * 1.4426950408889634f);
  t.s += acc;
}

template <bool VEC>
__global__ __launch_bounds__(256) void k_vocab_gate(VocabGateArgs a) {
  const int row = blockIdx.x;
  const int b = row / a.n_rows;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint16_t* x = a.logits + (int64_t)row * a.V;

  TopState t{-INFINITY, 0.f, INT_MAX};
  if constexpr (VEC) {
    const int nch = a.V >> 3;
    const int mchunk = a.mask_id >> 3, mlane = a.mask_id & 7;
    int c = tid;
    for (; c + 256 < nch; c += 512) {  // two independent 16-byte loads in flight
      const u32x4_t w0 = *reinterpret_cast<const u32x4_t*>(x + (int64_t)c * 8);
      const u32x4_t w1 = *reinterpret_cast<const u32x4_t*>(x + (int64_t)(c + 256) * 8);
      float v[8];
      v[0] = bf16_bits_to_f32(w0.x & 0xffff); v[1] = bf16_bits_to_f32(w0.x >> 16);
      v[2] = bf16_bits_to_f32(w0.y & 0xffff); v[3] = bf16_bits_to_f32(w0.y >> 16);
      v[4] = bf16_bits_to_f32(w0.z & 0xffff); v[5] = bf16_bits_to_f32(w0.z >> 16);
      v[6] = bf16_bits_to_f32(w0.w & 0xffff); v[7] = bf16_bits_to_f32(w0.w >> 16);
      if (c == mchunk) v[mlane] = -INFINITY;
      consume8(t, v, c * 8);
      v[0] = bf16_bits_to_f32(w1.x & 0xffff); v[1] = bf16_bits_to_f32(w1.x >> 16);
      v[2] = bf16_bits_to_f32(w1.y & 0xffff); v[3] = bf16_bits_to_f32(w1.y >> 16);
      v[4] = bf16_bits_to_f32(w1.z & 0xffff); v[5] = bf16_bits_to_f32(w1.z >> 16);
      v[6] = bf16_bits_to_f32(w1.w & 0xffff); v[7] = bf16_bits_to_f32(w1.w >> 16);
      if (c + 256 == mchunk) v[mlane] = -INFINITY;
      consume8(t, v, (c + 256) * 8);
    }
    for (; c < nch; c += 256) {
      const u32x4_t w0 = *reinterpret_cast<const u32x4_t*>(x + (int64_t)c * 8);
      float v[8];
      v[0] = bf16_bits_to_f32(w0.x & 0xffff); v[1] = bf16_bits_to_f32(w0.x >> 16);
      v[2] = bf16_bits_to_f32(w0.y & 0xffff); v[3] = bf16_bits_to_f32(w0.y >> 16);
      v[4] = bf16_bits_to_f32(w0.z & 0xffff); v[5] = bf16_bits_to_f32(w0.z >> 16);
      v[6] = bf16_bits_to_f32(w0.w & 0xffff); v[7] = bf16_bits_to_f32(w0.w >> 16);
      if (c == mchunk) v[mlane] = -INFINITY;
      consume8(t, v, c * 8);
    }
  } else {
    for (int v = tid; v < a.V; v += 256) {
      if (v == a.mask_id) continue;
      const float f = bf16_bits_to_f32(x[v]);
      if (f > t.m) {
        t.s = t.m == -INFINITY ? 0.f : t.s * exp2f((t.m - f) * 1.4426950408889634f);
        t.m = f;
        t.arg = v;
      }
      t.s += exp2f((f - t.m) * 1.4426950408889634f);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    TopState u;
    u.m = __shfl_xor(t.m, o, 64);
    u.s = __shfl_xor(t.s, o, 64);
    u.arg = __shfl_xor(t.arg, o, 64);
    t = merge(t, u);
  }
  __shared__ float sm_m[4], sm_s[4];
  __shared__ int sm_a[4];
  __shared__ int is_last;
  if (lane == 0) { sm_m[wave] = t.m; sm_s[wave] = t.s; sm_a[wave] = t.arg; }
  __syncthreads();
  if (tid == 0) {
    TopState r{sm_m[0], sm_s[0], sm_a[0]};
    for (int w = 1; w < 4; ++w) r = merge(r, TopState{sm_m[w], sm_s[w], sm_a[w]});
    // agent-coherent (sc1) stores instead of a release fence, which would write back the
    // whole L2: once they complete (vmcnt 0) they are visible to the last workgroup
    __hip_atomic_store(&a.top1[row], r.arg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&a.conf[row], 1.0f / r.s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);
    const int old =
        __hip_atomic_fetch_add(&a.tickets[b], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    is_last = (old == a.n_rows - 1);
  }
  __syncthreads();
  if (!is_last) return;

  // ---- phase 2: decision rules for batch row b --------------------------------------
  const int BL = a.block_len;
  const int blk = a.block_idx[b];
  const int s = a.step_idx[b];
  if (tid == 0) __hip_atomic_store(&a.tickets[b], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (blk < 0 || s < 0) {  // malformed state: touch nothing outside the scored rows
    if (tid == 0) a.done[b] = 0;
    return;
  }
  if (blk >= a.n_blocks) {  // row already finished
    if (tid < BL) a.decision[(int64_t)b * BL + tid] = 0;
    if (tid == 0) a.done[b] = 1;
    return;
  }
  const int lo = a.prompt_len + blk * BL;
  const int row0 = a.row_begin >= 0 ? a.row_begin : lo;
  const bool act = tid < BL;
  const int64_t gi = (int64_t)b * a.L + lo + tid;

  __shared__ float sc[CORA_MAX_BLOCK];
  __shared__ int su[CORA_MAX_BLOCK];
  int U = 0, xh = 0, m = 0;
  float c = 0.f;
  if (act) {
    U = a.unresolved[gi];
    const int64_t ri = (int64_t)b * a.n_rows + (lo + tid - row0);
    xh = __hip_atomic_load(&a.top1[ri], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    c = __hip_atomic_load(&a.conf[ri], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int prev = s == 0 ? -1 : a.prev_top1[gi];
    int mm = s == 0 ? 0 : a.persist[gi];
    if (U) {                                              // Eq. (2)
      mm = (prev != -1 && prev == xh) ? mm + 1 : 0;
      prev = xh;
    }
    if (s == 0 || U) { a.prev_top1[gi] = prev; a.persist[gi] = mm; }
    m = mm;
    sc[tid] = c;
    su[tid] = U;
  }
  __syncthreads();
  const int S = a.steps_per_block;
  const int k = a.k_transfer >= 0 ? a.k_transfer : BL / S + (s < BL % S ? 1 : 0);
  bool T = false, A = false;
  if (act && U) {
    int rank = 0;
    for (int j = 0; j < BL; ++j)
      rank += (su[j] && (sc[j] > c || (sc[j] == c && j < tid))) ? 1 : 0;
    T = rank < k;                                         // transfer rule
    A = !T && a.gate_enabled && c >= a.delta_p && m >= a.m_req;   // Eq. (3)
    if (T || A) {                                         // Eq. (4)
      a.tokens[gi] = xh;
      a.unresolved[gi] = 0;
    }
  }
  if (act) a.decision[(int64_t)b * BL + tid] = T ? 1 : (A ? 2 : 0);
  const int left = __syncthreads_or(act && U && !(T || A));
  if (tid == 0) {
    if (a.passes) a.passes[(int64_t)b * a.n_blocks + blk] += 1;
    if (!left) {
      a.block_idx[b] = blk + 1;
      a.step_idx[b] = 0;
    } else {
      a.step_idx[b] = s + 1;
    }
    a.done[b] = left ? 0 : 1;
  }
}

hipError_t launch_vocab_gate(const VocabGateArgs& a, hipStream_t s) {
  const int rows = a.B * a.n_rows;
  if (rows == 0) return hipSuccess;
  if (a.V % 8 == 0)
    hipLaunchKernelGGL(k_vocab_gate<true>, dim3(rows), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k_vocab_gate<false>, dim3(rows), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace cora
