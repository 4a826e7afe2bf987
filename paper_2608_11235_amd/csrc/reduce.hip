// Consumers of split-K partials (EPI_PART_F32 GEMMs): the partials of an output are added
// in split order, so the result does not depend on scheduling, and the sum goes straight
// into what the next kernel reads.
#include "common.hpp"
#include "internal.hpp"

namespace cora {

// One workgroup per row: fold the split-K partials of a residual GEMM into h (in split
// order, so the sum does not depend on scheduling), then normalise the updated row for the
// next GEMM.  Row values stay in registers between the two phases.  SPLITS, the threads NT
// and the chunk count C (float4 chunks per thread, C * NT * 4 >= d) are compile-time, so
// every partial and residual load of a thread is issued before the first add; rows of
// 4096 take 1024 threads with one chunk each, which keeps the most loads in flight.
template <int SPLITS, int C, int NT>
__global__ __launch_bounds__(NT) void k_residual_norm(float* __restrict__ h,
                                                      const float* __restrict__ part,
                                                      int64_t slab, int d,
                                                      const float* __restrict__ w,
                                                      uint16_t* __restrict__ out, float eps) {
  const int64_t r = blockIdx.x;
  float* x = h + r * d;
  const float* p = part + r * d;
  float4 pv[C][SPLITS], v[C];
#pragma unroll
  for (int i = 0; i < C; ++i) {
    const int c = (threadIdx.x + i * NT) * 4;
    if (c < d) {
#pragma unroll
      for (int sp = 0; sp < SPLITS; ++sp) pv[i][sp] = *reinterpret_cast<const float4*>(p + sp * slab + c);
      v[i] = *reinterpret_cast<const float4*>(x + c);
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < C; ++i) {
    const int c = (threadIdx.x + i * NT) * 4;
    if (c < d) {
      float4 acc = pv[i][0];
#pragma unroll
      for (int sp = 1; sp < SPLITS; ++sp) {
        acc.x += pv[i][sp].x;
        acc.y += pv[i][sp].y;
        acc.z += pv[i][sp].z;
        acc.w += pv[i][sp].w;
      }
      v[i].x += acc.x;
      v[i].y += acc.y;
      v[i].z += acc.z;
      v[i].w += acc.w;
      *reinterpret_cast<float4*>(x + c) = v[i];
      ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    }
  }
  if (!out) return;
  ss = warp_sum(ss);
  __shared__ float red[NT / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) tot += red[i];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  uint16_t* o = out + r * d;
#pragma unroll
  for (int i = 0; i < C; ++i) {
    const int c = (threadIdx.x + i * NT) * 4;
    if (c < d) {
      const float4 g = *reinterpret_cast<const float4*>(w + c);
      u32x2_t q;
      q.x = pack_bf16x2(v[i].x * inv * g.x, v[i].y * inv * g.y);
      q.y = pack_bf16x2(v[i].z * inv * g.z, v[i].w * inv * g.w);
      *reinterpret_cast<u32x2_t*>(o + c) = q;
    }
  }
}

template <int SPLITS>
static void residual_norm_c(int d4, dim3 grid, hipStream_t s, float* h, const float* part,
                            int64_t slab, int d, const float* w, uint16_t* out, float eps) {
#define RN(C_, NT_) hipLaunchKernelGGL((k_residual_norm<SPLITS, C_, NT_>), grid, dim3(NT_), 0, s, h, part, slab, d, w, out, eps)
  if (d4 <= 256) RN(1, 256);
  else if (d4 <= 512) RN(1, 512);
  else if (d4 <= 1024) RN(1, 1024);
  else RN(2, 1024);
#undef RN
}

hipError_t launch_residual_norm(float* h, const float* part, int splits, int rows, int d,
                                const float* w, uint16_t* out, float eps, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (d % 4 != 0 || d > RESIDUAL_NORM_MAX_D) return hipErrorInvalidValue;
  static_assert(RESIDUAL_NORM_MAX_D <= 2 * 1024 * 4, "at most 2 float4 chunks per thread");
  const int d4 = d / 4;
  const int64_t slab = (int64_t)rows * d;
  const dim3 grid(rows);
  switch (splits) {
    case 1: residual_norm_c<1>(d4, grid, s, h, part, slab, d, w, out, eps); break;
    case 2: residual_norm_c<2>(d4, grid, s, h, part, slab, d, w, out, eps); break;
    case 4: residual_norm_c<4>(d4, grid, s, h, part, slab, d, w, out, eps); break;
    case 8: residual_norm_c<8>(d4, grid, s, h, part, slab, d, w, out, eps); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// QKV projection partials -> q and k with rotate-half RoPE, v transposed.  q/k columns are
// pair-interleaved within a head, so a thread's 4 columns (4x .. 4x+3, inside one head) are
// two RoPE pairs; it handles the rows 4y .. 4y+3 (all 16-byte partial loads issued before
// the first add), and for v writes each column's 4 positions as one vector when they fall in
// one sequence.
template <int SPLITS>
__global__ __launch_bounds__(256) void k_qkv_finish(const float* __restrict__ part, int M, int N,
                                                    const float* __restrict__ bias, QkvOut o) {
  const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (c >= N) return;
  const int r0 = blockIdx.y * 4;
  const int nr = M - r0 < 4 ? M - r0 : 4;
  const int64_t slab = (int64_t)M * N;
  const int hd = o.head_dim, half = hd / 2;
  const int hq = o.n_heads * hd, hkv = o.n_kv_heads * hd;
  const int sec = c < hq ? 0 : (c < hq + hkv ? 1 : 2);
  const int cc = c - (sec == 0 ? 0 : (sec == 1 ? hq : hq + hkv));
  const int head = cc / hd, pd = cc % hd;
  const float4 bv = bias ? *reinterpret_cast<const float4*>(bias + c) : float4{0.f, 0.f, 0.f, 0.f};
  float4 pv[4][SPLITS];
#pragma unroll
  for (int t = 0; t < 4; ++t)
    if (t < nr) {
#pragma unroll
      for (int sp = 0; sp < SPLITS; ++sp)
        pv[t][sp] = *reinterpret_cast<const float4*>(part + sp * slab + (int64_t)(r0 + t) * N + c);
    }
  float x[4][4] = {};  // [row][column]; rows past M stay zero and are not stored
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t >= nr) continue;
    float4 v = pv[t][0];
#pragma unroll
    for (int sp = 1; sp < SPLITS; ++sp) {
      v.x += pv[t][sp].x;
      v.y += pv[t][sp].y;
      v.z += pv[t][sp].z;
      v.w += pv[t][sp].w;
    }
    x[t][0] = v.x + bv.x;
    x[t][1] = v.y + bv.y;
    x[t][2] = v.z + bv.z;
    x[t][3] = v.w + bv.w;
  }
  int b = r0 / o.L, pos = r0 - b * o.L;
  if (sec == 2 && nr == 4 && (o.L & 3) == 0) {  // pos % 4 == 0: all four rows in sequence b
    uint16_t* dst = o.vt + ((int64_t)(b * o.n_kv_heads + head) * hd + pd) * o.Ls + pos;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      u32x2_t q;
      q.x = pack_bf16x2(x[0][j], x[1][j]);
      q.y = pack_bf16x2(x[2][j], x[3][j]);
      *reinterpret_cast<u32x2_t*>(dst + j * o.Ls) = q;
    }
    return;
  }
  if (sec < 2) {
    // every row's cos/sin loads are issued before the first store: a load behind a store
    // would wait for that store too
    int bt[4], pt[4];
    float2 cs[4], sn[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      bt[t] = b;
      pt[t] = pos;
      if (t < nr) {
        cs[t] = *reinterpret_cast<const float2*>(o.cos_t + pos * half + (pd >> 1));
        sn[t] = *reinterpret_cast<const float2*>(o.sin_t + pos * half + (pd >> 1));
      }
      if (++pos == o.L) {
        pos = 0;
        ++b;
      }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (t >= nr) break;
      u32x2_t q;
      q.x = pack_bf16x2(x[t][0] * cs[t].x - x[t][1] * sn[t].x, x[t][1] * cs[t].x + x[t][0] * sn[t].x);
      q.y = pack_bf16x2(x[t][2] * cs[t].y - x[t][3] * sn[t].y, x[t][3] * cs[t].y + x[t][2] * sn[t].y);
      uint16_t* dst = sec == 0 ? o.q + ((int64_t)(bt[t] * o.n_heads + head) * o.Ls + pt[t]) * hd
                               : o.k + ((int64_t)(bt[t] * o.n_kv_heads + head) * o.Ls + pt[t]) * hd;
      *reinterpret_cast<u32x2_t*>(dst + pd) = q;
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t >= nr) break;
    {
      uint16_t* dst = o.vt + ((int64_t)(b * o.n_kv_heads + head) * hd + pd) * o.Ls + pos;
#pragma unroll
      for (int j = 0; j < 4; ++j) dst[j * o.Ls] = (uint16_t)f32_to_bf16_bits(x[t][j]);
    }
    if (++pos == o.L) {
      pos = 0;
      ++b;
    }
  }
}

hipError_t launch_qkv_finish(const float* part, int splits, int M, int N, const float* bias,
                             const QkvOut& o, hipStream_t s) {
  if (M == 0) return hipSuccess;
  if (N % 4 != 0 || o.head_dim % 4 != 0) return hipErrorInvalidValue;
  const dim3 grid((N / 4 + 255) / 256, (M + 3) / 4);
#define QF(S_) hipLaunchKernelGGL((k_qkv_finish<S_>), grid, dim3(256), 0, s, part, M, N, bias, o)
  switch (splits) {
    case 1: QF(1); break;
    case 2: QF(2); break;
    case 4: QF(4); break;
    case 8: QF(8); break;
    default: return hipErrorInvalidValue;
  }
#undef QF
  return hipGetLastError();
}

}  // namespace cora
