// Initial window scores from prompt attention (Sec. 4.2: prompt attention
// initialises the window scores before the first tier assignment).
//
// The observation queries are the last n_obs prompt positions.  For KV head g
// of sequence b their rows are r = h_local * n_obs + j (h_local < H_q / H_kv,
// j < n_obs; query position T - n_obs + j), a contiguous [rows][d] slab of the
// [B][H_q][n_obs][d] query tensor.  Row r attends causally to keys 0 .. its
// position.  The window score is the mass the window's keys receive, summed
// over rows and KV heads and divided by H_q.
//
// Four launches, all reductions in a fixed order (bitwise repeatable):
//   k_obs_pass<false>  per block of 256 keys: row max / exp-sum of the block
//   k_obs_rows         per row: global max M and 1 / L over the blocks
//   k_obs_pass<true>   per block: probabilities exp(x - M) / L summed over rows,
//                      one mass per key
//   k_obs_windows      per window: key masses summed over KV heads and tokens
//
// Logits come from 16x16x32 bf16 MFMAs with the keys as the A operand (rows =
// 16 keys) and the query rows as the B operand (columns = 16 query rows): a
// lane holds 4 keys of one query row, so row statistics fold in-lane and then
// over the lanes l, l ^ 16, l ^ 32, and key masses fold over the 16 lanes of a
// row group.  Each wave owns 64 keys of the block (their A operands stay in
// registers for every row); the query rows are staged in LDS, 128 at a time.
#include "qv_device.h"

namespace qv {

constexpr int kObsKeys = 256;          // keys per workgroup
constexpr int kObsWaveKeys = 64;       // keys per wave (4 MFMA tiles)
constexpr int kObsChunk = 128;         // query rows staged in LDS at once
constexpr int kObsRowBytes = 272;      // 256 B of a row + 16 B pad (conflict-free B reads)

__device__ __forceinline__ f32x4 mfma_obs(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// four workgroups per compute unit (at most 128 VGPRs) for the statistics
// pass, three for the mass pass, which also keeps 16 per-key sums per lane
template <bool MASS>
constexpr int obs_waves_per_simd() { return MASS ? 3 : 4; }

template <bool MASS>
__global__ __launch_bounds__(256, obs_waves_per_simd<MASS>()) void k_obs_pass(ObsArgs a) {
  const int blk = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T, n_rows = a.n_rows;
  const int lr = lane & 15, lq = lane >> 4;
  __shared__ __attribute__((aligned(16))) uint8_t sq[kObsChunk * kObsRowBytes];
  __shared__ float2 sst[4][kObsChunk];   // per wave row statistics (pass 1) / row M, 1/L (pass 2)

  const uint16_t* qb = a.q + ((int64_t)b * a.H_q + (int64_t)g * a.gqa) * a.n_obs * kHeadDim;
  // this wave's 64 keys as A operands: tile kt, k-step kc covers channels
  // 32 kc + 8 lq .. + 7 of key key0 + 16 kt + lr
  const int key0 = blk * kObsKeys + wave * kObsWaveKeys;
  const uint16_t* kb = a.k + ((int64_t)b * a.H_kv + g) * T * kHeadDim;
  u32x4 kop[4][4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    const int key = key0 + 16 * kt + lr;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
      kop[kt][kc] = key < T ? *(const u32x4*)(kb + (int64_t)key * kHeadDim + 32 * kc + 8 * lq)
                            : (u32x4){0, 0, 0, 0};
  }
  const int pos0 = T - a.n_obs;   // position of observation row j = pos0 + j
  float colacc[4][4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) colacc[kt][i] = 0.f;

  for (int r0 = 0; r0 < n_rows; r0 += kObsChunk) {
    const int nr = min(kObsChunk, n_rows - r0);
    __syncthreads();   // the previous chunk's rows and statistics are consumed
#pragma unroll 2
    for (int i = 0; i < kObsChunk * 16 / 256; ++i) {
      const int c = tid + 256 * i, row = c >> 4, part = c & 15;
      const u32x4 v = row < nr ? *(const u32x4*)(qb + (int64_t)(r0 + row) * kHeadDim + 8 * part)
                               : (u32x4){0, 0, 0, 0};
      *(u32x4*)(sq + row * kObsRowBytes + 16 * part) = v;
    }
    if (MASS && tid < kObsChunk)
      sst[0][tid] = tid < nr ? a.row_ml[((int64_t)b * a.H_kv + g) * n_rows + r0 + tid]
                             : make_float2(INFINITY, 0.f);   // padding rows add exp2(-inf) * 0
    __syncthreads();
    for (int rt = 0; rt < (nr + 15) / 16; ++rt) {
      const int row = rt * 16 + lr;            // this lane's query row inside the chunk
      const int rg = r0 + row;
      const int pos = pos0 + (rg % a.n_obs);
      f32x4 acc[4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) acc[kt] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        const u32x4 qv = *(const u32x4*)(sq + row * kObsRowBytes + 64 * kc + 16 * lq);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
          acc[kt] = mfma_obs(__builtin_bit_cast(bf16x8, kop[kt][kc]), __builtin_bit_cast(bf16x8, qv),
                             acc[kt]);
      }
      // acc[kt][i]: raw logit of key key0 + 16 kt + 4 lq + i for this row.  Only
      // a wave whose keys pass the first observation position (or the prompt's
      // end) masks keys, to -inf; rows past the chunk's end are never read
      // back (pass 1) or have 1 / L = 0 (pass 2)
      if (key0 + kObsWaveKeys - 1 > pos0) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = key0 + 16 * kt + 4 * lq + i;
            if (key >= T || key > pos) acc[kt][i] = -INFINITY;
          }
      }
      const float sc = a.scale_log2;
      if (!MASS) {
        float mr = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) mr = fmaxf(mr, acc[kt][i]);
        const float m = mr * sc;   // log2 units
        float l = 0.f;
        if (mr > -INFINITY) {
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) l += __builtin_amdgcn_exp2f(fmaf(acc[kt][i], sc, -m));
        }
        float mc = m, lc = l;
#pragma unroll
        for (int o = 16; o <= 32; o <<= 1) {
          const float m2 = __shfl_xor(mc, o, 64), l2 = __shfl_xor(lc, o, 64);
          const float mm = fmaxf(mc, m2);
          float ls = 0.f;
          if (mc > -INFINITY) ls += lc * __builtin_amdgcn_exp2f(mc - mm);
          if (m2 > -INFINITY) ls += l2 * __builtin_amdgcn_exp2f(m2 - mm);
          mc = mm;
          lc = ls;
        }
        if (lq == 0) sst[wave][row] = make_float2(mc, lc);
      } else {
        // (M, 1 / L) of this row (log2 units; M finite for every real row, since
        // key 0 is visible to all of them); masked logits add exp2(-inf) = 0
        const float2 ml = sst[0][row];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            colacc[kt][i] = fmaf(__builtin_amdgcn_exp2f(fmaf(acc[kt][i], sc, -ml.x)), ml.y, colacc[kt][i]);
      }
    }
    if (!MASS) {
      // the four waves' statistics of each row, folded in wave order
      __syncthreads();
      if (tid < nr) {
        float m = -INFINITY, l = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float2 s = sst[w][tid];
          const float mm = fmaxf(m, s.x);
          float ls = 0.f;
          if (m > -INFINITY) ls += l * __builtin_amdgcn_exp2f(m - mm);
          if (s.x > -INFINITY) ls += s.y * __builtin_amdgcn_exp2f(s.x - mm);
          m = mm;
          l = ls;
        }
        a.blk_ml[(((int64_t)b * a.H_kv + g) * n_rows + r0 + tid) * a.n_blk + blk] = make_float2(m, l);
      }
    }
  }
  if (MASS) {
    // sum over the 16 query rows of each lane group (lanes with the same lq)
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v = colacc[kt][i];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
        colacc[kt][i] = v;
      }
    if (lr == 0) {
      float* out = a.key_mass + ((int64_t)b * a.H_kv + g) * a.T_pad;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
        *(float4*)(out + key0 + 16 * kt + 4 * lq) =
            make_float4(colacc[kt][0], colacc[kt][1], colacc[kt][2], colacc[kt][3]);
    }
  }
}

// (M, 1 / L) of every row from its blocks' (max, exp-sum) pairs; one wave per row,
// lane j folds blocks j, j + 64, ... then a butterfly in a fixed order
__global__ __launch_bounds__(64) void k_obs_rows(ObsArgs a) {
  const int r = blockIdx.x, g = blockIdx.y, b = blockIdx.z, lane = threadIdx.x;
  const float2* st = a.blk_ml + (((int64_t)b * a.H_kv + g) * a.n_rows + r) * a.n_blk;
  float m = -INFINITY, l = 0.f;
  for (int k = lane; k < a.n_blk; k += 64) {
    const float2 s = st[k];
    const float mm = fmaxf(m, s.x);
    float ls = 0.f;
    if (m > -INFINITY) ls += l * __builtin_amdgcn_exp2f(m - mm);
    if (s.x > -INFINITY) ls += s.y * __builtin_amdgcn_exp2f(s.x - mm);
    m = mm;
    l = ls;
  }
  for (int o = 1; o < 64; o <<= 1) {
    const float m2 = __shfl_xor(m, o, 64), l2 = __shfl_xor(l, o, 64);
    const float mm = fmaxf(m, m2);
    float ls = 0.f;
    if (m > -INFINITY) ls += l * __builtin_amdgcn_exp2f(m - mm);
    if (m2 > -INFINITY) ls += l2 * __builtin_amdgcn_exp2f(m2 - mm);
    m = mm;
    l = ls;
  }
  if (lane == 0)
    a.row_ml[((int64_t)b * a.H_kv + g) * a.n_rows + r] = make_float2(m, l > 0.f ? 1.f / l : 0.f);
}

// score[b][w] = (1 / H_q) * (sum of the key masses of the window's tokens over
// all KV heads); one wave per window: lane j folds entries j, j + 64, ... of
// the (head, token) list, then a butterfly (a fixed order)
__global__ __launch_bounds__(256) void k_obs_windows(ObsArgs a) {
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6), b = blockIdx.y, lane = threadIdx.x & 63;
  if (w >= a.n_w) return;   // uniform per wave
  const int t0 = a.sink + w * a.W, nt = min(a.W, a.T - t0);
  const float* km = a.key_mass + (int64_t)b * a.H_kv * a.T_pad + t0;
  float s = 0.f;
  for (int e = lane; e < a.H_kv * a.W; e += 64) {
    const int g = e / a.W, t = e % a.W;
    if (t < nt) s += km[(int64_t)g * a.T_pad + t];
  }
  for (int o = 1; o < 64; o <<= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) a.scores[(int64_t)b * a.n_w + w] = s / (float)a.H_q;
}

hipError_t launch_prefill_scores(const ObsArgs& a, hipStream_t st) {
  const dim3 grid(a.n_blk, a.H_kv, a.B);
  hipLaunchKernelGGL(k_obs_pass<false>, grid, dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_obs_rows, dim3(a.n_rows, a.H_kv, a.B), dim3(64), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_obs_pass<true>, grid, dim3(256), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.n_w > 0) hipLaunchKernelGGL(k_obs_windows, dim3((a.n_w + 3) / 4, a.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace qv
