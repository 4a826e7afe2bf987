// Bidirectional (non-causal) attention for gfx950, online softmax in fp32.
//
// Inputs: q [B, H, Ls, hd], k [B, Hkv, Ls, hd] (RoPE applied), vt [B, Hkv, hd, Ls]
// (v transposed), rows >= L zero.  Output: o [B * L, H * hd] bf16.
// One workgroup = 64 queries of one head (4 wavefronts x 16 queries) times SPLIT parts of
// the key range: with SPLIT = 2 a second group of 4 wavefronts runs the same queries over
// the second half of the key tiles, and the partial softmax states (max, sum, O) are merged
// through LDS at the end, in part order.  Small grids use SPLIT = 2: at most two
// workgroups per CU at hd 128, fewer than two at hd 64, counted for the model's max_batch
// (the choice is made for the rows a launch is planned for, not the live ones, so that a
// row's rounding never depends on its batch).
// Two kernels share the arithmetic:
//  - k_attention_dl (hd 128, the model shapes) fetches the 64-key K and V^T tiles straight
//    into LDS with 16-byte buffer loads that write LDS (no staging registers), which keeps
//    a wavefront in 128 registers: four wavefronts per SIMD.
//  - k_attention (hd 64) stages the next tile in registers while the current one is
//    multiplied out of LDS.
// Within a tile, the K fragments are read in two batches of 8 (one LDS round trip per
// batch rather than one per MFMA pair).
// Softmax terms use the hardware v_exp_f32; results below 2^-126 flush to zero, which no
// sum holding its max term can notice.  The running reference max of each query is moved
// (and O and the sum rescaled) only when a tile's max exceeds it by more than 2^8, so exp
// arguments are <= 8 and most tiles skip the rescale; the common factor cancels in the final
// O / l.  The lane groups of a query exchange their maxima only on such tiles.  The
// 1/sqrt(hd) scale (times log2 e) is folded into one FMA per score, and the tile's key mask
// is applied only on a partial last tile (a scalar branch).
// Everything is computed transposed with v_mfma_f32_16x16x32_bf16 so that a query's
// softmax statistics never leave its lanes:
//   S^T = K Q^T   (A = K tile from LDS, B = Q^T held in registers)
//   O^T = V^T P^T (A = V^T tile from LDS, B = P^T straight from the S^T registers)
// Feeding the S^T registers as P^T fixes the key order of a 32-key MFMA step; the K tile's
// rows are stored in a permuted key order (see krow) so that this order is 8 consecutive
// keys per lane group, and each V^T fragment is a single 16-byte LDS read.
// A 16-byte LDS read serves the 32 lanes of each wavefront half from one 512-byte bank
// window, so the 16-byte slots (address / 16 mod 32) those lanes touch must be distinct.
// k_attention pads its rows to 18 (K) and 10 (V^T) slots, which puts the 16 rows x 2 column
// chunks of a half-wavefront on 32 distinct slots (odd strides such as 17 and 9 give
// two-way conflicts on every read); k_attention_dl permutes the chunks of unpadded rows.
// Workgroups are dealt to the 8 XCDs round-robin; the (head, query tile) order is remapped
// so that each XCD runs a contiguous range of heads, whose K/V tiles then stay in its L2.
#include "common.hpp"
#include "internal.hpp"

namespace cora {

// Register-staged kernel (hd 64): the next tile's loads are in flight in registers while
// the current tile is multiplied out of LDS.  Small grids double-buffer the tile (one
// barrier per tile); large grids (SB) keep one LDS tile buffer and at most 168 registers, so
// three workgroups share a CU.
template <int HD, int SPLIT, bool SB = false>
__global__ __launch_bounds__(256 * SPLIT, SB && SPLIT == 1 ? 3 : 1) void k_attention(const uint16_t* __restrict__ q,
                                                   const uint16_t* __restrict__ k,
                                                   const uint16_t* __restrict__ vt,
                                                   uint16_t* __restrict__ out, int L, int Ls,
                                                   int H, int Hkv, float scale_log2) {
  constexpr int KT = 64;          // keys per tile
  constexpr int LDKS = HD + 16;   // padded LDS rows
  constexpr int LDVS = KT + 16;
  constexpr int CK = KT * HD / 8 / 256;  // 16-byte chunks per thread per tile (K and V^T each)
  constexpr int NB = SB ? 1 : 2;  // LDS tile buffers
  // K tiles [NB][SPLIT][KT * LDKS], then V^T tiles [NB][SPLIT][HD * LDVS], in one region
  // that the merge of the parts reuses after the last tile
  constexpr int KSZ = KT * LDKS, VSZ = HD * LDVS;
  __shared__ __attribute__((aligned(16))) uint16_t lds[NB * SPLIT * (KSZ + VSZ)];
  auto Kt = [&](int buf, int p) { return lds + (buf * SPLIT + p) * KSZ; };
  auto Vt = [&](int buf, int p) { return lds + NB * SPLIT * KSZ + (buf * SPLIT + p) * VSZ; };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // which part of the key range (wave-uniform, so tile indices and branches stay scalar)
  const int part = __builtin_amdgcn_readfirstlane(wave >> 2);
  const int tl = tid & 255, tpart = part;    // loader thread: its index and part
  // (head, query tile) of this workgroup: contiguous ranges per XCD
  const int li = xcd_remap(blockIdx.x + blockIdx.y * gridDim.x, gridDim.x * gridDim.y);
  const int qt = li % gridDim.x, bh = li / gridDim.x;
  const int b = bh / H, h = bh % H, kvh = h / (H / Hkv);
  const int q0 = qt * 64 + (wave & 3) * 16;
  const int g = lane >> 4, r16 = lane & 15;

  const uint16_t* qh = q + ((int64_t)(b * H + h) * Ls) * HD;
  const uint16_t* kh = k + ((int64_t)(b * Hkv + kvh) * Ls) * HD;
  const uint16_t* vh = vt + ((int64_t)(b * Hkv + kvh) * HD) * Ls;

  bf16x8_t qf[HD / 32];
#pragma unroll
  for (int kk = 0; kk < HD / 32; ++kk)
    qf[kk] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(qh + (int64_t)(q0 + r16) * HD + kk * 32 + g * 8));

  f32x4_t o[HD / 16];
#pragma unroll
  for (int d = 0; d < HD / 16; ++d) o[d] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_ref = -INFINITY, l_part = 0.f;  // reference max (log2 units) and sum of this lane
  constexpr float SLACK = 8.f;            // exp arguments stay <= SLACK

  // K tile [64 keys][HD] and V^T tile [HD][64 keys] of part tpart, read through buffer
  // resources over this head's K and V^T: each chunk has a fixed per-lane byte offset and a
  // tile adds the uniform key0 * HD * 2 (K) or key0 * 2 (V^T) as the scalar offset
  u32x4_t rk[CK], rv[CK];
  const __amdgpu_buffer_rsrc_t k_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)kh, (short)0, Ls * HD * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t v_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)vh, (short)0, HD * Ls * 2, 0x00020000);
  // chunk i of this thread: K row tl / (HD/8) + i * (256 / (HD/8)), V^T row tl / (KT/8) +
  // i * (256 / (KT/8))
  int kvo[CK], vvo[CK];
#pragma unroll
  for (int i = 0; i < CK; ++i) {
    kvo[i] = ((tl / (HD / 8) + i * (256 / (HD / 8))) * HD + (tl % (HD / 8)) * 8) * 2;
    vvo[i] = ((tl / (KT / 8) + i * (256 / (KT / 8))) * Ls + (tl % (KT / 8)) * 8) * 2;
  }
  auto fetch = [&](int key0) {
#pragma unroll
    for (int i = 0; i < CK; ++i) {
      rk[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(k_rs, kvo[i], key0 * HD * 2, 0));
      rv[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(v_rs, vvo[i], key0 * 2, 0));
    }
  };
  // K rows are stored in a permuted key order: tile key k = 32 a + 8 g + 4 b + i (a, b in
  // {0, 1}, g < 4, i < 4) goes to LDS row (2 a + b) * 16 + 4 g + i.  S^T block kb then holds,
  // in lane group g, keys 32 (kb / 2) + 8 g + 4 (kb % 2) + i, so the 8 P^T slots of lane
  // group g in key step ks are the 8 consecutive keys 32 ks + 8 g .. + 7 and the matching
  // V^T fragment is one 16-byte read of the natural V^T layout.
  auto krow = [](int k) { return ((k >> 5) * 2 + ((k >> 2) & 1)) * 16 + ((k >> 3) & 3) * 4 + (k & 3); };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CK; ++i) {
      const int c = tl + i * 256;
      const int kr = c / (HD / 8), kc = (c % (HD / 8)) * 8;
      *reinterpret_cast<u32x4_t*>(Kt(buf, tpart) + krow(kr) * LDKS + kc) = rk[i];
      const int vr = c / (KT / 8), vc = (c % (KT / 8)) * 8;
      *reinterpret_cast<u32x4_t*>(Vt(buf, tpart) + vr * LDVS + vc) = rv[i];
    }
  };

  // part p owns key tiles [p * per, min((p + 1) * per, n_tiles)); step j works on tile
  // p * per + j of every part, and parts that ran out skip the work but keep the barriers.
  const int n_tiles = (L + KT - 1) / KT;
  const int per = (n_tiles + SPLIT - 1) / SPLIT;
  const bool load0 = tpart * per < n_tiles;
  if (load0) fetch(tpart * per * KT);
  stash(0);
  __syncthreads();
  for (int j = 0; j < per; ++j) {
    const int buf = SB ? 0 : (j & 1), kt = part * per + j, key0 = kt * KT;
    const int next = tpart * per + j + 1;  // this thread's next tile to load
    if (j + 1 < per && next < n_tiles) fetch(next * KT);  // in flight during this tile
    if (kt < n_tiles) {
      // K fragments are requested in two batches of 8 (two 16-key blocks each), each
      // batch before its MFMAs: two LDS round trips per tile, in 32 registers
      f32x4_t st[4];
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        bf16x8_t kf[2][HD / 32];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int kk = 0; kk < HD / 32; ++kk)
            kf[kb][kk] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(
                Kt(buf, part) + ((2 * hb + kb) * 16 + r16) * LDKS + kk * 32 + g * 8));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) st[2 * hb + kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < HD / 32; ++kk)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
            st[2 * hb + kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kb][kk], qf[kk], st[2 * hb + kb], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      // the first key step's V^T fragments are requested before the softmax
      u32x4_t vf[HD / 16];
#pragma unroll
      for (int d = 0; d < HD / 16; ++d)
        vf[d] = *reinterpret_cast<const u32x4_t*>(Vt(buf, part) + (d * 16 + r16) * LDVS + g * 8);
      __builtin_amdgcn_sched_barrier(0);
      if (key0 + KT > L) {  // partial last tile (scalar branch): keys past L drop out
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = key0 + 32 * (kb >> 1) + 8 * g + 4 * (kb & 1) + i;
            if (key >= L) st[kb][i] = -INFINITY;
          }
      }
      float lmax = -INFINITY;  // this lane's max of raw scores (the scale is positive)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) lmax = fmaxf(lmax, st[kb][i]);
      // the lane groups of a query exchange their maxima only when some lane holds a score
      // beyond its query's reference by more than SLACK; otherwise no reference moves
      if (__any(lmax * scale_log2 > m_ref + SLACK)) {
        float tmax = fmaxf(lmax, __shfl_xor(lmax, 16, 64));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
        const float tm = tmax * scale_log2;
        const bool grow = tm > m_ref + SLACK;  // true on a lane's first tile (m_ref = -inf)
        const float m_new = grow ? tm : m_ref;
        const float alpha = fast_exp2(m_ref - m_new);  // 1 where kept, 0 while m_ref is -inf
        m_ref = m_new;
        l_part *= alpha;
#pragma unroll
        for (int d = 0; d < HD / 16; ++d) o[d] *= alpha;
      }
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = fast_exp2(fmaf(st[kb][i], scale_log2, -m_ref));
          st[kb][i] = p;
          l_part += p;
        }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        u32x4_t pb;
        pb.x = pack_bf16x2(st[2 * ks][0], st[2 * ks][1]);
        pb.y = pack_bf16x2(st[2 * ks][2], st[2 * ks][3]);
        pb.z = pack_bf16x2(st[2 * ks + 1][0], st[2 * ks + 1][1]);
        pb.w = pack_bf16x2(st[2 * ks + 1][2], st[2 * ks + 1][3]);
        const bf16x8_t bfrag = as_bf16x8(pb);
        if (ks == 1) {
#pragma unroll
          for (int d = 0; d < HD / 16; ++d)
            vf[d] = *reinterpret_cast<const u32x4_t*>(Vt(buf, part) + (d * 16 + r16) * LDVS + 32 + g * 8);
          __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int d = 0; d < HD / 16; ++d)
          o[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vf[d]), bfrag, o[d], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if (j + 1 < per) {
      if constexpr (SB) __syncthreads();  // one buffer: every wavefront is done with tile j
      stash(SB ? 0 : buf ^ 1);
    }
    __syncthreads();
  }

  if constexpr (SPLIT >= 2) {
    // parts 1 .. SPLIT-1 hand their (max, partial sums, O) to part 0's wavefronts, which
    // fold them in part order; the tiles' LDS is free after the loop's last barrier
    constexpr int NF = 2 + 4 * (HD / 16);
    float* comb = reinterpret_cast<float*>(lds);
    static_assert(sizeof(lds) >= (size_t)(SPLIT - 1) * 4 * NF * 64 * sizeof(float), "merge buffer");
    if (part > 0) {
      const int slot = ((part - 1) * 4 + (wave & 3)) * NF * 64 + lane;
      comb[slot] = m_ref;
      comb[slot + 64] = l_part;
#pragma unroll
      for (int d = 0; d < HD / 16; ++d)
#pragma unroll
        for (int i = 0; i < 4; ++i) comb[slot + (2 + 4 * d + i) * 64] = o[d][i];
    }
    __syncthreads();
    if (part > 0) return;
#pragma unroll
    for (int p = 1; p < SPLIT; ++p) {
      const int slot = ((p - 1) * 4 + (wave & 3)) * NF * 64 + lane;
      const float m1 = comb[slot], l1 = comb[slot + 64];
      const float m = fmaxf(m_ref, m1);
      const float a0 = fast_exp2(m_ref - m), a1 = fast_exp2(m1 - m);
      m_ref = m;
      l_part = l_part * a0 + l1 * a1;
#pragma unroll
      for (int d = 0; d < HD / 16; ++d)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          o[d][i] = o[d][i] * a0 + comb[slot + (2 + 4 * d + i) * 64] * a1;
    }
  }

  float l = l_part;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  const float inv = 1.0f / l;
  const int qi = q0 + r16;
  if (qi < L) {
    uint16_t* dst = out + ((int64_t)b * L + qi) * ((int64_t)H * HD) + h * HD;
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) {
      u32x2_t p;
      p.x = pack_bf16x2(o[d][0] * inv, o[d][1] * inv);
      p.y = pack_bf16x2(o[d][2] * inv, o[d][3] * inv);
      *reinterpret_cast<u32x2_t*>(dst + d * 16 + g * 4) = p;
    }
  }
}

// Direct-to-LDS kernel (hd 128): a wavefront's 16-byte buffer load with the LDS flag writes
// 64 consecutive 16-byte slots of LDS, so the tiles are unpadded and each row's 16-byte
// chunks are permuted instead, by an XOR with bits of the row index (K: row & 15, V^T:
// (row >> 1) & 7); the fragment reads of every half-wavefront then land on 32 distinct
// slots.  The K rows hold the permuted key order of krow above.  A workgroup holds SPLIT x
// 32 KB of LDS (one K and one V^T buffer per part), and four wavefronts share each SIMD.
// Two barriers per tile: after the S^T MFMAs and the softmax, every wavefront's V^T loads
// have landed and the K buffer is free, so the next K tile is fetched while V^T is read and
// multiplied; after the O^T MFMAs the next V^T tile is fetched while K is.
template <int HD, int SPLIT>
__global__ __launch_bounds__(256 * SPLIT) __attribute__((amdgpu_waves_per_eu(4, 4))) void k_attention_dl(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ vt,
    uint16_t* __restrict__ out, int L, int Ls, int H, int Hkv, float scale_log2) {
  static_assert(HD == 128, "16 chunks per K row");
  constexpr int KT = 64;
  constexpr int KROW = HD * 2, VROW = KT * 2;  // bytes per K row and per V^T row
  constexpr int KBYTES = KT * KROW, VBYTES = HD * VROW, PBYTES = KBYTES + VBYTES;
  __shared__ __attribute__((aligned(16))) unsigned char lds[SPLIT * PBYTES];
  typedef __attribute__((address_space(3))) void* lds_ptr_t;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int part = wave >> 2, w4 = wave & 3;  // key-range part, wavefront within the part
  const int li = xcd_remap(blockIdx.x + blockIdx.y * gridDim.x, gridDim.x * gridDim.y);
  const int qt = li % gridDim.x, bh = li / gridDim.x;
  const int b = bh / H, h = bh % H, kvh = h / (H / Hkv);
  const int q0 = qt * 64 + w4 * 16;
  const int g = lane >> 4, r16 = lane & 15;
  unsigned char* const pl = lds + part * PBYTES;  // this part's K and V^T tiles

  const uint16_t* qh = q + ((int64_t)(b * H + h) * Ls) * HD;
  const uint16_t* kh = k + ((int64_t)(b * Hkv + kvh) * Ls) * HD;
  const uint16_t* vh = vt + ((int64_t)(b * Hkv + kvh) * HD) * Ls;
  const __amdgpu_buffer_rsrc_t k_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)kh, (short)0, Ls * HD * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t v_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)vh, (short)0, HD * Ls * 2, 0x00020000);

  // this lane's slot in each of the wavefront's 4 K and 4 V^T loads of a tile: load t of
  // wavefront w4 fills slots [64 (4 w4 + t), + 64) of its part's tile
  int kvo[4], vvo[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int R = (w4 * 4 + t) * 4 + (lane >> 4), c = (lane & 15) ^ (R & 15);
    const int key = (R >> 5) * 32 + ((R >> 2) & 3) * 8 + ((R >> 4) & 1) * 4 + (R & 3);  // krow^-1
    kvo[t] = (key * HD + c * 8) * 2;
    const int Rv = (w4 * 4 + t) * 8 + (lane >> 3), cv = (lane & 7) ^ ((Rv >> 1) & 7);
    vvo[t] = (Rv * Ls + cv * 8) * 2;
  }
  auto fetch_k = [&](int key0) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(k_rs, (lds_ptr_t)(pl + (w4 * 4 + t) * 1024), 16, kvo[t],
                                               key0 * HD * 2, 0, 0);
  };
  auto fetch_v = [&](int key0) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(v_rs, (lds_ptr_t)(pl + KBYTES + (w4 * 4 + t) * 1024), 16,
                                               vvo[t], key0 * 2, 0, 0);
  };

  // part p owns key tiles [p * per, min((p + 1) * per, n_tiles)); parts that run out skip
  // the work but keep the barriers
  const int n_tiles = (L + KT - 1) / KT;
  const int per = (n_tiles + SPLIT - 1) / SPLIT;
  const int t0 = part * per, t1 = t0 + per < n_tiles ? t0 + per : n_tiles;

  bf16x8_t qf[HD / 32];
#pragma unroll
  for (int kk = 0; kk < HD / 32; ++kk)
    qf[kk] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(qh + (int64_t)(q0 + r16) * HD + kk * 32 + g * 8));
  if (t0 < t1) {
    fetch_k(t0 * KT);
    fetch_v(t0 * KT);
  }
  f32x4_t o[HD / 16];
#pragma unroll
  for (int d = 0; d < HD / 16; ++d) o[d] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_ref = -INFINITY, l_part = 0.f;
  constexpr float SLACK = 8.f;

  // fragment read addresses: K chunk kk * 4 + g of row kb * 16 + r16 sits at slot
  // (kk * 4 + g) ^ r16 of its row; V^T chunk ks * 4 + g of row d * 16 + r16 at slot
  // (ks * 4 + g) ^ (r16 >> 1)
  int kra[HD / 32], vra[2];
#pragma unroll
  for (int kk = 0; kk < HD / 32; ++kk) kra[kk] = part * PBYTES + r16 * KROW + (((kk * 4 + g) ^ r16) & 15) * 16;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
    vra[ks] = part * PBYTES + KBYTES + r16 * VROW + (((ks * 4 + g) ^ (r16 >> 1)) & 7) * 16;

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
  for (int kk = 0; kk < HD / 32; ++kk) asm volatile("" ::"v"(qf[kk]));  // Q is in before the loop
  __syncthreads();
  for (int j = 0; j < per; ++j) {
    const int kt = t0 + j, key0 = kt * KT;
    const bool live = kt < t1;  // wave-uniform
    f32x4_t st[4];
    if (live) {
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        bf16x8_t kf[2][HD / 32];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int kk = 0; kk < HD / 32; ++kk)
            kf[kb][kk] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(lds + kra[kk] + (2 * hb + kb) * 16 * KROW));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) st[2 * hb + kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < HD / 32; ++kk)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
            st[2 * hb + kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kb][kk], qf[kk], st[2 * hb + kb], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if (live) {
      if (key0 + KT > L) {  // partial last tile (scalar branch): keys past L drop out
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = key0 + 32 * (kb >> 1) + 8 * g + 4 * (kb & 1) + i;
            if (key >= L) st[kb][i] = -INFINITY;
          }
      }
      float lmax = -INFINITY;  // this lane's max of raw scores (the scale is positive)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) lmax = fmaxf(lmax, st[kb][i]);
      if (__any(lmax * scale_log2 > m_ref + SLACK)) {
        float tmax = fmaxf(lmax, __shfl_xor(lmax, 16, 64));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
        const float tm = tmax * scale_log2;
        const bool grow = tm > m_ref + SLACK;
        const float m_new = grow ? tm : m_ref;
        const float alpha = fast_exp2(m_ref - m_new);
        m_ref = m_new;
        l_part *= alpha;
#pragma unroll
        for (int d = 0; d < HD / 16; ++d) o[d] *= alpha;
      }
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = fast_exp2(fmaf(st[kb][i], scale_log2, -m_ref));
          st[kb][i] = p;
          l_part += p;
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (kt + 1 < t1) fetch_k(key0 + KT);
    if (live) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        u32x4_t vf[HD / 16];
#pragma unroll
        for (int d = 0; d < HD / 16; ++d)
          vf[d] = *reinterpret_cast<const u32x4_t*>(lds + vra[ks] + d * 16 * VROW);
        __builtin_amdgcn_sched_barrier(0);
        u32x4_t pb;
        pb.x = pack_bf16x2(st[2 * ks][0], st[2 * ks][1]);
        pb.y = pack_bf16x2(st[2 * ks][2], st[2 * ks][3]);
        pb.z = pack_bf16x2(st[2 * ks + 1][0], st[2 * ks + 1][1]);
        pb.w = pack_bf16x2(st[2 * ks + 1][2], st[2 * ks + 1][3]);
        const bf16x8_t bfrag = as_bf16x8(pb);
#pragma unroll
        for (int d = 0; d < HD / 16; ++d)
          o[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vf[d]), bfrag, o[d], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // every wavefront is done reading V^T and its K loads have landed: after the barrier
    // the next K tile is whole and the V^T buffer is free
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (kt + 1 < t1) fetch_v(key0 + KT);
  }

  if constexpr (SPLIT >= 2) {
    // parts 1 .. SPLIT-1 hand their (max, partial sums, O) to part 0's wavefronts, which
    // fold them in part order; the tiles' LDS is free after the loop's last barrier
    constexpr int NF = 2 + 4 * (HD / 16);
    float* comb = reinterpret_cast<float*>(lds);
    static_assert(sizeof(lds) >= (size_t)(SPLIT - 1) * 4 * NF * 64 * sizeof(float), "merge buffer");
    if (part > 0) {
      const int slot = ((part - 1) * 4 + w4) * NF * 64 + lane;
      comb[slot] = m_ref;
      comb[slot + 64] = l_part;
#pragma unroll
      for (int d = 0; d < HD / 16; ++d)
#pragma unroll
        for (int i = 0; i < 4; ++i) comb[slot + (2 + 4 * d + i) * 64] = o[d][i];
    }
    __syncthreads();
    if (part > 0) return;
#pragma unroll
    for (int p = 1; p < SPLIT; ++p) {
      const int slot = ((p - 1) * 4 + w4) * NF * 64 + lane;
      const float m1 = comb[slot], l1 = comb[slot + 64];
      const float m = fmaxf(m_ref, m1);
      const float a0 = fast_exp2(m_ref - m), a1 = fast_exp2(m1 - m);
      m_ref = m;
      l_part = l_part * a0 + l1 * a1;
#pragma unroll
      for (int d = 0; d < HD / 16; ++d)
#pragma unroll
        for (int i = 0; i < 4; ++i) o[d][i] = o[d][i] * a0 + comb[slot + (2 + 4 * d + i) * 64] * a1;
    }
  }

  float l = l_part;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  const float inv = 1.0f / l;
  const int qi = q0 + r16;
  if (qi < L) {
    uint16_t* dst = out + ((int64_t)b * L + qi) * ((int64_t)H * HD) + h * HD;
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) {
      u32x2_t p;
      p.x = pack_bf16x2(o[d][0] * inv, o[d][1] * inv);
      p.y = pack_bf16x2(o[d][2] * inv, o[d][3] * inv);
      *reinterpret_cast<u32x2_t*>(dst + d * 16 + g * 4) = p;
    }
  }
}

hipError_t launch_attention(const uint16_t* q, const uint16_t* k, const uint16_t* vt,
                            uint16_t* out, int B, int L, int Ls, int H, int Hkv, int hd,
                            int plan_B, int num_cus, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (plan_B < B) return hipErrorInvalidValue;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
  const dim3 grid(Ls / 64, B * H);
  const bool split = (int64_t)grid.x * plan_B * H < 2 * (int64_t)num_cus;
#define ATTN(HD_, SP_, SB_)                                                                \
  hipLaunchKernelGGL((k_attention<HD_, SP_, SB_>), grid, dim3(256 * SP_), 0, s, q, k, vt, out, L, \
                     Ls, H, Hkv, scale_log2)
  if (hd == 128) {
    // two key-range parts while the planned grid has at most two workgroups per CU (four
    // parts, measured, lose to two: each part's pipeline would run only a few tiles)
    const int64_t wgs = (int64_t)grid.x * plan_B * H;
#define ATTN_DL(SP_) \
  hipLaunchKernelGGL((k_attention_dl<128, SP_>), grid, dim3(256 * SP_), 0, s, q, k, vt, out, L, Ls, H, Hkv, \
                     scale_log2)
    if (wgs <= 2 * (int64_t)num_cus) ATTN_DL(2);
    else ATTN_DL(1);
#undef ATTN_DL
  } else if (hd == 64) {
    if (split) ATTN(64, 2, false);
    else ATTN(64, 1, true);
  } else {
    return hipErrorInvalidValue;
  }
#undef ATTN
  return hipGetLastError();
}

}  // namespace cora
