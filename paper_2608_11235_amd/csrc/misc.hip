// Weight init (counter-based generator), embedding gather, RMSNorm and decode-state init.
#include "common.hpp"
#include "internal.hpp"

namespace cora {

// ---- counter-based N(0, std) generator ---------------------------------------------------
// SplitMix64 finaliser; the stream started at key = mix(seed) yields outputs 2c+1 and 2c+2
// for counter c = (tensor_id << 40) | element; Box-Muller in fp64; round to fp32 then bf16.
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ULL;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBULL;
  z ^= z >> 31;
  return z;
}

__device__ __forceinline__ float normal_from_counter(uint64_t key, uint64_t ctr, double std_dev) {
  const uint64_t G = 0x9E3779B97F4A7C15ULL;
  const uint64_t h1 = mix64(key + (2 * ctr + 1) * G);
  const uint64_t h2 = mix64(key + (2 * ctr + 2) * G);
  const double u1 = (double)((h1 >> 11) + 1) * 0x1.0p-53;
  const double u2 = (double)(h2 >> 11) * 0x1.0p-53;
  const double n = sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925286766559 * u2);
  return (float)(std_dev * n);
}

// element (pr, c) of the physical matrix goes to pr * ld + c, or, packed (ld % 64 == 0), to
// block (pr / 64, c / 64) of 64 x 64 (row-major inside), blocks ordered by row block then
// column block
__device__ __forceinline__ int64_t packed64_index(int64_t pr, int64_t c, int64_t ld) {
  return ((pr >> 6) * (ld >> 6) + (c >> 6)) * 4096 + (pr & 63) * 64 + (c & 63);
}

__global__ void k_init_bf16(uint16_t* __restrict__ dst, uint64_t key, uint64_t base, int64_t rows,
                            int64_t cols, int64_t ld, int row_map, int64_t row_offset,
                            double std_dev, int hd, int packed) {
  for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
    int64_t pr;
    if (row_map == ROW_GATE) pr = (r >> 5) * 64 + (r & 31);
    else if (row_map == ROW_UP) pr = (r >> 5) * 64 + 32 + (r & 31);
    else if (row_map == ROW_ROPE_PAIR) pr = row_offset + (r / hd) * hd + rope_pair_pos((int)(r % hd), hd);
    else pr = row_offset + r;
    for (int64_t c = threadIdx.x; c < cols; c += blockDim.x) {
      const uint64_t ctr = base | (uint64_t)(r * cols + c);
      dst[packed ? packed64_index(pr, c, ld) : pr * ld + c] =
          (uint16_t)f32_to_bf16_bits(normal_from_counter(key, ctr, std_dev));
    }
  }
}

// bias vectors: drawn like any tensor, rounded to bf16, stored as fp32
__global__ void k_init_f32(float* __restrict__ dst, uint64_t key, uint64_t base, int64_t n,
                           double std_dev, int pair_hd) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    const float v = normal_from_counter(key, base | (uint64_t)e, std_dev);
    const int64_t pe = pair_hd > 0 ? (e / pair_hd) * pair_hd + rope_pair_pos((int)(e % pair_hd), pair_hd) : e;
    dst[pe] = bf16_bits_to_f32(f32_to_bf16_bits(v));
  }
}

__global__ void k_fill_f32(float* dst, float v, int64_t n) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x)
    dst[e] = v;
}

static uint64_t host_mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ULL;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBULL;
  z ^= z >> 31;
  return z;
}

hipError_t launch_init_bf16(uint16_t* dst, uint64_t seed, uint64_t tensor_id, int64_t rows,
                            int64_t cols, int64_t ld, int row_map, int64_t row_offset, double std_dev,
                            int head_dim, hipStream_t s, bool packed) {
  if (packed && ld % 64 != 0) return hipErrorInvalidValue;
  const int grid = (int)(rows < 16384 ? rows : 16384);
  hipLaunchKernelGGL(k_init_bf16, dim3(grid), dim3(256), 0, s, dst, host_mix64(seed),
                     tensor_id << 40, rows, cols, ld, row_map, row_offset, std_dev, head_dim,
                     packed ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_init_f32(float* dst, uint64_t seed, uint64_t tensor_id, int64_t n,
                           double std_dev, int pair_head_dim, hipStream_t s) {
  const int grid = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(k_init_f32, dim3(grid), dim3(256), 0, s, dst, host_mix64(seed),
                     tensor_id << 40, n, std_dev, pair_head_dim);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* dst, float v, int64_t n, hipStream_t s) {
  const int grid = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(k_fill_f32, dim3(grid), dim3(256), 0, s, dst, v, n);
  return hipGetLastError();
}

// ---- embedding: h[m, :] = E[tokens[m], :] (fp32 residual stream) ------------------------
__global__ void k_embed(const int32_t* __restrict__ tokens, const uint16_t* __restrict__ E,
                        float* __restrict__ h, int d, int V) {
  const int m = blockIdx.x;
  const int tok = min(max(tokens[m], 0), V - 1);  // out-of-range ids never read outside E
  const uint16_t* src = E + (int64_t)tok * d;
  float* dst = h + (int64_t)m * d;
  for (int c = threadIdx.x * 8; c < d; c += blockDim.x * 8) {
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(src + c);
    float4 lo, hi;
    lo.x = bf16_bits_to_f32(v.x & 0xffff); lo.y = bf16_bits_to_f32(v.x >> 16);
    lo.z = bf16_bits_to_f32(v.y & 0xffff); lo.w = bf16_bits_to_f32(v.y >> 16);
    hi.x = bf16_bits_to_f32(v.z & 0xffff); hi.y = bf16_bits_to_f32(v.z >> 16);
    hi.z = bf16_bits_to_f32(v.w & 0xffff); hi.w = bf16_bits_to_f32(v.w >> 16);
    *reinterpret_cast<float4*>(dst + c) = lo;
    *reinterpret_cast<float4*>(dst + c + 4) = hi;
  }
}

hipError_t launch_embed(const int32_t* tokens, const uint16_t* E, float* h, int M, int d, int V,
                        hipStream_t s) {
  if (M == 0) return hipSuccess;
  hipLaunchKernelGGL(k_embed, dim3(M), dim3(256), 0, s, tokens, E, h, d, V);
  return hipGetLastError();
}

// ---- RMSNorm: fp32 rows in, bf16 rows out ------------------------------------------------
__global__ __launch_bounds__(256) void k_rmsnorm(const float* __restrict__ h,
                                                 const float* __restrict__ w,
                                                 uint16_t* __restrict__ out, int d, float eps,
                                                 RowSel sel) {
  const int j = blockIdx.x;
  int64_t src = j;
  if (sel.mode != 0) {
    const int b = j / sel.n_rows, r = j % sel.n_rows;
    int base = sel.row_begin;
    if (sel.mode == 2) {
      int blk = sel.block_idx[b];
      blk = max(0, min(blk, sel.n_blocks - 1));
      base = sel.prompt_len + blk * sel.block_len;
    }
    src = (int64_t)b * sel.L + base + r;
  }
  const float* x = h + src * d;
  float ss = 0.f;
  for (int c = threadIdx.x * 4; c < d; c += 256 * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = warp_sum(ss);
  __shared__ float part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = part[0] + part[1] + part[2] + part[3];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  uint16_t* o = out + (int64_t)j * d;
  for (int c = threadIdx.x * 4; c < d; c += 256 * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + c);
    const float4 g = *reinterpret_cast<const float4*>(w + c);
    u32x2_t p;
    p.x = pack_bf16x2(v.x * inv * g.x, v.y * inv * g.y);
    p.y = pack_bf16x2(v.z * inv * g.z, v.w * inv * g.w);
    *reinterpret_cast<u32x2_t*>(o + c) = p;
  }
}

hipError_t launch_rmsnorm(const float* h, const float* w, uint16_t* out, int rows, int d,
                          float eps, RowSel sel, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(k_rmsnorm, dim3(rows), dim3(256), 0, s, h, w, out, d, eps, sel);
  return hipGetLastError();
}

// ---- decode state: canvas = prompt ++ masks --------------------------------------------
__global__ void k_state_init(const int32_t* __restrict__ prompt, int B, int P, int G, int mask_id,
                             int32_t* tokens, uint8_t* unresolved, int32_t* prev, int32_t* persist,
                             int32_t* block_idx, int32_t* step_idx, int32_t* passes,
                             int n_blocks) {
  const int L = P + G;
  const int64_t n = (int64_t)B * L;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int b = (int)(e / L), i = (int)(e % L);
    tokens[e] = i < P ? prompt[(int64_t)b * P + i] : mask_id;
    unresolved[e] = i < P ? 0 : 1;
    prev[e] = -1;
    persist[e] = 0;
    if (i == 0) {
      block_idx[b] = 0;
      step_idx[b] = 0;
      if (passes)
        for (int j = 0; j < n_blocks; ++j) passes[(int64_t)b * n_blocks + j] = 0;
    }
  }
}

hipError_t launch_state_init(const int32_t* prompt, int B, int P, int G, int mask_id,
                             int32_t* tokens, uint8_t* unresolved, int32_t* prev, int32_t* persist,
                             int32_t* block_idx, int32_t* step_idx, int32_t* passes, int n_blocks,
                             hipStream_t s) {
  const int64_t n = (int64_t)B * (P + G);
  const int grid = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
  hipLaunchKernelGGL(k_state_init, dim3(grid), dim3(256), 0, s, prompt, B, P, G, mask_id, tokens,
                     unresolved, prev, persist, block_idx, step_idx, passes, n_blocks);
  return hipGetLastError();
}

// ---- batch-row compaction of a decode state ----------------------------------------------
// dst row i <- src row map[i] (tokens, unresolved, previous top-1, counters, block and step
// index, passes per block); one workgroup per destination row.
__global__ void k_gather_state(DecodeRows src, DecodeRows dst, const int32_t* __restrict__ map,
                               int L, int n_blocks) {
  const int i = blockIdx.x, r = map[i];
  const int64_t so = (int64_t)r * L, dof = (int64_t)i * L;
  for (int e = threadIdx.x; e < L; e += blockDim.x) {
    dst.tokens[dof + e] = src.tokens[so + e];
    dst.unresolved[dof + e] = src.unresolved[so + e];
    dst.prev[dof + e] = src.prev[so + e];
    dst.persist[dof + e] = src.persist[so + e];
  }
  for (int j = threadIdx.x; j < n_blocks; j += blockDim.x)
    dst.passes[(int64_t)i * n_blocks + j] = src.passes[(int64_t)r * n_blocks + j];
  if (threadIdx.x == 0) {
    dst.block_idx[i] = src.block_idx[r];
    dst.step_idx[i] = src.step_idx[r];
  }
}

hipError_t launch_gather_state(const DecodeRows& src, const DecodeRows& dst, const int32_t* map,
                               int n, int L, int n_blocks, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_state, dim3(n), dim3(256), 0, s, src, dst, map, L, n_blocks);
  return hipGetLastError();
}

// Final tokens and passes of the rows rows[i] of a (compacted) state go to row orig[i] of the
// outputs.
__global__ void k_scatter_rows(const int32_t* __restrict__ tokens, const int32_t* __restrict__ passes,
                               const int32_t* __restrict__ rows, const int32_t* __restrict__ orig,
                               int L, int n_blocks, int32_t* __restrict__ out_tokens,
                               int32_t* __restrict__ out_passes) {
  const int r = rows[blockIdx.x], o = orig[blockIdx.x];
  for (int e = threadIdx.x; e < L; e += blockDim.x)
    out_tokens[(int64_t)o * L + e] = tokens[(int64_t)r * L + e];
  for (int j = threadIdx.x; j < n_blocks; j += blockDim.x)
    out_passes[(int64_t)o * n_blocks + j] = passes[(int64_t)r * n_blocks + j];
}

hipError_t launch_scatter_rows(const int32_t* tokens, const int32_t* passes, const int32_t* rows,
                               const int32_t* orig, int n, int L, int n_blocks,
                               int32_t* out_tokens, int32_t* out_passes, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_scatter_rows, dim3(n), dim3(256), 0, s, tokens, passes, rows, orig, L,
                     n_blocks, out_tokens, out_passes);
  return hipGetLastError();
}

}  // namespace cora
