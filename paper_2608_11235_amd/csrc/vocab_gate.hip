// Vocab reduction over logits rows, and the decision rules.  A denoising step computes
// Eq. (1) inside its LM-head pass and runs only k_gate_rules from here; k_vocab_top1
// reduces logits a caller hands over (cora_vocab_gate), and the rows of a step whose
// vocabulary is too small to hold the fused pass's partials in the logits buffer.
//
// k_vocab_top1, one workgroup per logits row: a single coalesced pass over the bf16 row
// (16-byte streaming loads, the next group of four in flight while the current one is
// consumed) keeps a running (max, sum of exp(l - max)) per thread and the chunk that first
// reached the max (its raw words kept in registers), merged across the wavefront with xor
// shuffles and across the 4 wavefronts through LDS in a fixed order, so results are
// bitwise reproducible.  The row's top-1 token is the lowest id among equal maxima, the
// mask id is skipped, and the confidence is c = max softmax = 1 / sum_v exp(l_v - l_max)
// (Eq. 1).
//
// k_gate_rules, one workgroup per batch row, on that row's active block (the kernel
// boundary orders it after every row's top-1 and confidence):
//   block step 0 -> previous top-1 and counters reset (persistence is per block);
//   Eq. (2) counter update on unresolved positions;
//   transfer rule: the k highest-confidence unresolved positions (ties -> lower position);
//   Eq. (3) gate on the other unresolved positions (c >= delta_p and m >= m_req);
//   Eq. (4) commit of both sets; with the EOS-aware controller, the lowest committed EOS
//   of the generation region cuts the canvas (later unresolved positions resolved as EOS);
//   block done once no unresolved position is left, then the row moves to its next block
//   (or stops after an EOS cut).
// Splitting the two removes a per-row tail (agent-coherent result stores, their
// completion, a ticket round trip) from every workgroup of the bandwidth-bound first pass.
#include <limits.h>

#include <algorithm>

#include "common.hpp"
#include "internal.hpp"

namespace cora {

// raw words of the chunk that first reached the running max (VEC row loop)
struct BestChunk {
  uint32_t w0, w1, w2, w3;
};

// Running (max, sum of exp(l - max)) over a group of 32 logits (chunks i = 0..3 of 8): one
// max and one rescale per group, then exp2 of every logit relative to the running max.  The
// argmax is not tracked per element: the chunk that first raises the running max is
// remembered with its raw words (strict >, so the earliest chunk holding the maximum; the
// four chunk maxima fall out of the max tree) and searched once after the row.
__device__ __forceinline__ void consume32(TopState& t, BestChunk& best, const float (&v)[32],
                                          const u32x4_t (&w)[4], int c) {
  float cmx[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float m = v[8 * i];
#pragma unroll
    for (int j = 1; j < 8; ++j) m = fmaxf(m, v[8 * i + j]);
    cmx[i] = m;
  }
  const float cm = fmaxf(fmaxf(cmx[0], cmx[1]), fmaxf(cmx[2], cmx[3]));
  if (cm > t.m) {
    t.s = t.m == -INFINITY ? 0.f : t.s * fast_exp2((t.m - cm) * LOG2E);
    t.m = cm;
    const int i = cmx[0] == cm ? 0 : (cmx[1] == cm ? 1 : (cmx[2] == cm ? 2 : 3));
    const u32x4_t bw = i == 0 ? w[0] : (i == 1 ? w[1] : (i == 2 ? w[2] : w[3]));
    best = BestChunk{bw.x, bw.y, bw.z, bw.w};
    t.arg = c + 256 * i;
  }
  if (t.m == -INFINITY) return;
  const float ml = t.m * LOG2E;
  float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
  for (int j = 0; j < 32; j += 2) {
    acc0 += fast_exp2(fmaf(v[j], LOG2E, -ml));
    acc1 += fast_exp2(fmaf(v[j + 1], LOG2E, -ml));
  }
  t.s += acc0 + acc1;
}

// PART: workgroup blockIdx.x = row * sp.parts + part reduces vocab chunks [part * sp.chunks,
// (part + 1) * sp.chunks) of its row (entries, not chunks, when !VEC) and stores the partial
// (max, sum, lowest arg max) at sp.p*[blockIdx.x]; k_top1_merge folds a row's parts in vocab
// order.  Without PART one workgroup covers the whole row and writes top1 / conf.
template <bool VEC, bool PART>
__global__ __launch_bounds__(256) void k_vocab_top1(VocabGateArgs a, VocabSplit sp) {
  const int row = PART ? blockIdx.x / sp.parts : blockIdx.x;
  const int part = PART ? blockIdx.x - row * sp.parts : 0;
  const int b = row / a.n_rows;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint16_t* x = a.logits + (int64_t)row * a.V;

  TopState t{-INFINITY, 0.f, INT_MAX};  // VEC: t.arg is a chunk index until the row ends
  if constexpr (VEC) {
    // Thread tid reads chunks (16 bytes = 8 logits) tid + 256 i, in groups of 4: chunks
    // c, c + 256, c + 512, c + 768.  The next group's loads are in flight while the current
    // group is consumed.  Only a wavefront whose group holds the mask id's chunk (a scalar
    // test) applies the mask override.
    const int c_lo = PART ? part * sp.chunks : 0;
    const int nch = PART ? min(c_lo + sp.chunks, a.V >> 3) : a.V >> 3;  // end of this range
    const int mchunk = a.mask_id >> 3, mlane = a.mask_id & 7;
    const u32x4_t* xv = reinterpret_cast<const u32x4_t*>(x);
    const u32x4_t NEG_INF4 = {0xff80ff80u, 0xff80ff80u, 0xff80ff80u, 0xff80ff80u};
    BestChunk best{0u, 0u, 0u, 0u};
    auto group = [&](const u32x4_t (&w)[4], int c) {
      float v[32];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[8 * i + 0] = bf16_bits_to_f32(w[i].x & 0xffff); v[8 * i + 1] = bf16_bits_to_f32(w[i].x >> 16);
        v[8 * i + 2] = bf16_bits_to_f32(w[i].y & 0xffff); v[8 * i + 3] = bf16_bits_to_f32(w[i].y >> 16);
        v[8 * i + 4] = bf16_bits_to_f32(w[i].z & 0xffff); v[8 * i + 5] = bf16_bits_to_f32(w[i].z >> 16);
        v[8 * i + 6] = bf16_bits_to_f32(w[i].w & 0xffff); v[8 * i + 7] = bf16_bits_to_f32(w[i].w >> 16);
      }
      const int cb = __builtin_amdgcn_readfirstlane(c - lane);  // chunk of lane 0
      const int dm = mchunk - cb;
      if (dm >= 0 && dm < 1024 && (dm & 255) < 64) {  // this wavefront's group holds the mask id
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (c + 256 * i == mchunk && j == mlane) v[8 * i + j] = -INFINITY;
      }
      consume32(t, best, v, w, c);
    };
    auto load4 = [&](u32x4_t (&w)[4], int c) {
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = __builtin_nontemporal_load(xv + c + 256 * i);
    };
    int c = c_lo + tid;
    if (c + 768 < nch) {
      // two register groups used alternately (no copies): one in flight, one consumed
      u32x4_t ga[4], gb[4];
      load4(ga, c);
      while (true) {
        if (c + 1024 + 768 >= nch) { group(ga, c); c += 1024; break; }
        load4(gb, c + 1024);
        group(ga, c);
        c += 1024;
        if (c + 1024 + 768 >= nch) { group(gb, c); c += 1024; break; }
        load4(ga, c + 1024);
        group(gb, c);
        c += 1024;
      }
    }
    if (c < nch) {  // at most 3 chunks left: one guarded group, missing chunks -inf
      u32x4_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = c + 256 * i < nch ? xv[c + 256 * i] : NEG_INF4;
      group(w, c);
    }
    // lowest index holding the max inside the remembered chunk (mask id excluded)
    if (t.m == -INFINITY) {
      t.arg = INT_MAX;
    } else {
      const int ch = t.arg;
      const uint32_t wd[4] = {best.w0, best.w1, best.w2, best.w3};
      int found = INT_MAX;
#pragma unroll
      for (int e = 7; e >= 0; --e) {
        const float f = bf16_bits_to_f32((e & 1) ? (wd[e >> 1] >> 16) : (wd[e >> 1] & 0xffff));
        if (f == t.m && !(ch == mchunk && e == mlane)) found = ch * 8 + e;
      }
      t.arg = found;
    }
  } else {
    const int v_lo = PART ? part * sp.chunks : 0;
    const int v_hi = PART ? min(v_lo + sp.chunks, a.V) : a.V;
    for (int v = v_lo + tid; v < v_hi; v += 256) {
      if (v == a.mask_id) continue;
      const float f = bf16_bits_to_f32(x[v]);
      if (f == -INFINITY) continue;
      if (f > t.m) {
        t.s = t.m == -INFINITY ? 0.f : t.s * fast_exp2((t.m - f) * LOG2E);
        t.m = f;
        t.arg = v;
      }
      t.s += fast_exp2((f - t.m) * LOG2E);
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
  if (lane == 0) { sm_m[wave] = t.m; sm_s[wave] = t.s; sm_a[wave] = t.arg; }
  __syncthreads();
  if (tid == 0) {
    TopState r{sm_m[0], sm_s[0], sm_a[0]};
    for (int w = 1; w < 4; ++w) r = merge(r, TopState{sm_m[w], sm_s[w], sm_a[w]});
    if constexpr (PART) {
      sp.pm[blockIdx.x] = r.m;
      sp.ps[blockIdx.x] = r.s;
      sp.pa[blockIdx.x] = r.arg;
    } else {
      const int64_t o = (int64_t)b * a.out_ld + a.out_off + (row - b * a.n_rows);
      a.top1[o] = r.arg;
      a.conf[o] = 1.0f / r.s;
    }
  }
}

__global__ __launch_bounds__(256) void k_gate_rules(VocabGateArgs a) {
  const int b = blockIdx.x, tid = threadIdx.x;
  const int BL = a.block_len;
  const int blk = a.block_idx[b];
  const int s = a.step_idx[b];
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
  const bool global = a.persist_scope == 1;
  if (global) {
    // Eq. (2) on the scored unresolved positions outside the active block (those inside
    // are updated below); counters run across blocks
    for (int j = tid; j < a.n_rows; j += blockDim.x) {
      const int p = row0 + j;
      if (p >= lo && p < lo + BL) continue;
      const int64_t g = (int64_t)b * a.L + p;
      if (!a.unresolved[g]) continue;
      const int x = a.top1[(int64_t)b * a.out_ld + j];
      const int pv = a.prev_top1[g];
      a.persist[g] = (pv != -1 && pv == x) ? a.persist[g] + 1 : 0;
      a.prev_top1[g] = x;
    }
  }

  __shared__ float sc[CORA_MAX_BLOCK];
  __shared__ int su[CORA_MAX_BLOCK];
  int U = 0, xh = 0, m = 0;
  float c = 0.f;
  if (act) {
    U = a.unresolved[gi];
    const int64_t ri = (int64_t)b * a.out_ld + (lo + tid - row0);
    xh = a.top1[ri];
    c = a.conf[ri];
    const bool reset = s == 0 && !global;                 // BLOCK scope: block becomes active
    int prev = reset ? -1 : a.prev_top1[gi];
    int mm = reset ? 0 : a.persist[gi];
    if (U) {                                              // Eq. (2)
      mm = (prev != -1 && prev == xh) ? mm + 1 : 0;
      prev = xh;
    }
    if (reset || U) { a.prev_top1[gi] = prev; a.persist[gi] = mm; }
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
  // EOS-aware controller: the lowest committed EOS of the generation region cuts the
  // canvas; later unresolved positions are resolved as EOS and the row stops after this
  // block
  __shared__ int s_cut;
  int cut = INT_MAX;
  if (a.eos_enabled) {
    if (tid == 0) s_cut = INT_MAX;
    __syncthreads();  // this step's commits are visible to the whole workgroup
    for (int p = a.prompt_len + tid; p < a.L; p += blockDim.x) {
      const int64_t g = (int64_t)b * a.L + p;
      if (!a.unresolved[g] && a.tokens[g] == a.eos_id) atomicMin(&s_cut, p);
    }
    __syncthreads();
    cut = s_cut;
    if (cut != INT_MAX) {
      for (int p = cut + 1 + tid; p < a.L; p += blockDim.x) {
        const int64_t g = (int64_t)b * a.L + p;
        if (a.unresolved[g]) {
          a.tokens[g] = a.eos_id;
          a.unresolved[g] = 0;
          if (p >= lo && p < lo + BL) a.decision[(int64_t)b * BL + (p - lo)] = 3;
        }
      }
    }
  }
  const bool cut_off = cut != INT_MAX && lo + tid > cut;
  const int left = __syncthreads_or(act && U && !(T || A) && !cut_off);
  if (tid == 0) {
    if (a.passes) a.passes[(int64_t)b * a.n_blocks + blk] += 1;
    if (!left) {
      a.block_idx[b] = cut != INT_MAX ? a.n_blocks : blk + 1;
      a.step_idx[b] = 0;
    } else {
      a.step_idx[b] = s + 1;
    }
    a.done[b] = left ? 0 : 1;
  }
}

hipError_t launch_vocab_top1(const VocabGateArgs& a, hipStream_t s) {
  const int rows = a.B * a.n_rows;
  if (rows == 0) return hipSuccess;
  const VocabSplit none{};
  if (a.V % 8 == 0)
    hipLaunchKernelGGL((k_vocab_top1<true, false>), dim3(rows), dim3(256), 0, s, a, none);
  else
    hipLaunchKernelGGL((k_vocab_top1<false, false>), dim3(rows), dim3(256), 0, s, a, none);
  return hipGetLastError();
}

int vocab_split_parts(int rows, int V, int num_cus, int64_t max_partials) {
  if (rows <= 0 || (int64_t)rows > max_partials) return 0;
  // each part keeps the 4-chunk load pipeline of every thread busy (>= 1024 chunks, or
  // 8192 entries without 16-byte chunks); enough parts for ~4 workgroups per CU
  const int units = V % 8 == 0 ? V / 8 : V;
  const int min_units = V % 8 == 0 ? 1024 : 8192;
  int parts = (4 * num_cus + rows - 1) / rows;
  parts = std::min(parts, std::max(1, units / min_units));
  parts = (int)std::min<int64_t>(parts, max_partials / rows);
  return std::max(parts, 1);
}

hipError_t launch_vocab_top1_split(const VocabGateArgs& a, const VocabSplit& in, hipStream_t s) {
  const int rows = a.B * a.n_rows;
  if (rows == 0) return hipSuccess;
  if (in.parts < 1 || !in.pm || !in.ps || !in.pa) return hipErrorInvalidValue;
  VocabSplit sp = in;
  const int units = a.V % 8 == 0 ? a.V / 8 : a.V;
  sp.chunks = (units + sp.parts - 1) / sp.parts;
  const dim3 grid((unsigned)((int64_t)rows * sp.parts));
  if (a.V % 8 == 0)
    hipLaunchKernelGGL((k_vocab_top1<true, true>), grid, dim3(256), 0, s, a, sp);
  else
    hipLaunchKernelGGL((k_vocab_top1<false, true>), grid, dim3(256), 0, s, a, sp);
  if (hipError_t e = hipGetLastError()) return e;
  return launch_top1_merge_parts(sp.pm, sp.ps, sp.pa, sp.parts, rows, a.n_rows, a.out_ld,
                                 a.out_off, a.top1, a.conf, s);
}

hipError_t launch_gate_rules(const VocabGateArgs& a, hipStream_t s) {
  if (a.B == 0) return hipSuccess;
  if (a.block_len > 256) return hipErrorInvalidValue;  // one thread per block position
  hipLaunchKernelGGL(k_gate_rules, dim3(a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace cora
