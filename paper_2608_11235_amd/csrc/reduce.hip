// Consumers of split-K partials (EPI_PART_F32 GEMMs): the partials of an output are added
// in split order, so the result does not depend on scheduling, and the sum goes straight
// into what the next kernel reads.
#include "common.hpp"
#include "internal.hpp"

namespace cora {

// One workgroup per row: fold the split-K partials of a residual GEMM into h (in split
// order, so the sum does not depend on scheduling), then normalise the updated row for the
// next GEMM.  Row values stay in registers between the two phases.
__global__ __launch_bounds__(256) void k_residual_norm(float* __restrict__ h,
                                                       const float* __restrict__ part,
                                                       int splits, int64_t slab, int d,
                                                       const float* __restrict__ w,
                                                       uint16_t* __restrict__ out, float eps) {
  constexpr int MAXC = RESIDUAL_NORM_MAX_D / 1024;  // float4 chunks per thread
  const int64_t r = blockIdx.x;
  float* x = h + r * d;
  const float* p = part + r * d;
  float4 v[MAXC];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = (threadIdx.x + i * 256) * 4;
    if (c < d) {
      float4 acc = *reinterpret_cast<const float4*>(p + c);
      for (int sp = 1; sp < splits; ++sp) {
        const float4 q = *reinterpret_cast<const float4*>(p + sp * slab + c);
        acc.x += q.x;
        acc.y += q.y;
        acc.z += q.z;
        acc.w += q.w;
      }
      float4 hv = *reinterpret_cast<const float4*>(x + c);
      hv.x += acc.x;
      hv.y += acc.y;
      hv.z += acc.z;
      hv.w += acc.w;
      *reinterpret_cast<float4*>(x + c) = hv;
      v[i] = hv;
      ss += hv.x * hv.x + hv.y * hv.y + hv.z * hv.z + hv.w * hv.w;
    }
  }
  if (!out) return;
  ss = warp_sum(ss);
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  uint16_t* o = out + r * d;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = (threadIdx.x + i * 256) * 4;
    if (c < d) {
      const float4 g = *reinterpret_cast<const float4*>(w + c);
      u32x2_t q;
      q.x = pack_bf16x2(v[i].x * inv * g.x, v[i].y * inv * g.y);
      q.y = pack_bf16x2(v[i].z * inv * g.z, v[i].w * inv * g.w);
      *reinterpret_cast<u32x2_t*>(o + c) = q;
    }
  }
}

hipError_t launch_residual_norm(float* h, const float* part, int splits, int rows, int d,
                                const float* w, uint16_t* out, float eps, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (splits < 1 || d % 4 != 0 || d > RESIDUAL_NORM_MAX_D) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_residual_norm, dim3(rows), dim3(256), 0, s, h, part, splits,
                     (int64_t)rows * d, d, w, out, eps);
  return hipGetLastError();
}

// QKV projection partials -> q and k with rotate-half RoPE, v transposed.  q/k columns are
// pair-interleaved within a head, so a thread's column pair (2x, 2x+1) is exactly one RoPE
// pair; it handles the rows 4y .. 4y+3, and for v writes the 4 positions as one vector when
// they fall in one sequence.
__global__ __launch_bounds__(256) void k_qkv_finish(const float* __restrict__ part, int splits,
                                                    int M, int N, const float* __restrict__ bias,
                                                    QkvOut o) {
  const int c = (blockIdx.x * 256 + threadIdx.x) * 2;
  if (c >= N) return;
  const int r0 = blockIdx.y * 4;
  const int nr = M - r0 < 4 ? M - r0 : 4;
  const int64_t slab = (int64_t)M * N;
  const int hd = o.head_dim, half = hd / 2;
  const int hq = o.n_heads * hd, hkv = o.n_kv_heads * hd;
  const int sec = c < hq ? 0 : (c < hq + hkv ? 1 : 2);
  const int cc = c - (sec == 0 ? 0 : (sec == 1 ? hq : hq + hkv));
  const int head = cc / hd, pd = cc % hd;
  const float b0 = bias ? bias[c] : 0.f, b1 = bias ? bias[c + 1] : 0.f;
  float x0[4], x1[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t < nr) {
      const float* p = part + (int64_t)(r0 + t) * N + c;
      float2 v = *reinterpret_cast<const float2*>(p);
      for (int sp = 1; sp < splits; ++sp) {
        const float2 q = *reinterpret_cast<const float2*>(p + sp * slab);
        v.x += q.x;
        v.y += q.y;
      }
      x0[t] = v.x + b0;
      x1[t] = v.y + b1;
    }
  }
  int b = r0 / o.L, pos = r0 - b * o.L;
  if (sec == 2 && nr == 4 && (o.L & 3) == 0) {  // pos % 4 == 0: all four rows in sequence b
    uint16_t* dst = o.vt + ((int64_t)(b * o.n_kv_heads + head) * hd + pd) * o.Ls + pos;
    u32x2_t v0, v1;
    v0.x = pack_bf16x2(x0[0], x0[1]);
    v0.y = pack_bf16x2(x0[2], x0[3]);
    v1.x = pack_bf16x2(x1[0], x1[1]);
    v1.y = pack_bf16x2(x1[2], x1[3]);
    *reinterpret_cast<u32x2_t*>(dst) = v0;
    *reinterpret_cast<u32x2_t*>(dst + o.Ls) = v1;
    return;
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t >= nr) break;
    if (sec < 2) {
      const float cs = o.cos_t[pos * half + (pd >> 1)], sn = o.sin_t[pos * half + (pd >> 1)];
      const float y0 = x0[t] * cs - x1[t] * sn, y1 = x1[t] * cs + x0[t] * sn;
      uint16_t* dst = sec == 0 ? o.q + ((int64_t)(b * o.n_heads + head) * o.Ls + pos) * hd
                               : o.k + ((int64_t)(b * o.n_kv_heads + head) * o.Ls + pos) * hd;
      *reinterpret_cast<uint32_t*>(dst + pd) = pack_bf16x2(y0, y1);
    } else {
      uint16_t* dst = o.vt + ((int64_t)(b * o.n_kv_heads + head) * hd + pd) * o.Ls + pos;
      dst[0] = (uint16_t)f32_to_bf16_bits(x0[t]);
      dst[o.Ls] = (uint16_t)f32_to_bf16_bits(x1[t]);
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
  if (splits < 1 || N % 2 != 0 || o.head_dim % 2 != 0) return hipErrorInvalidValue;
  const dim3 grid((N / 2 + 255) / 256, (M + 3) / 4);
  hipLaunchKernelGGL(k_qkv_finish, grid, dim3(256), 0, s, part, splits, M, N, bias, o);
  return hipGetLastError();
}

}  // namespace cora
