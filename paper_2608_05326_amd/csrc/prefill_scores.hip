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
// The keys are cut into chunks of 64 aligned with the windows: chunk c holds
// keys cbase + 64 c .. + 63, cbase = sink - 64 * ceil(sink / 64) <= 0, so a
// chunk is either all sink (and keys < 0) or exactly 64 / W whole windows.
// Three launches, every reduction in a fixed order (bitwise repeatable):
//   k_obs_chunks   one pass over the keys: per (row, chunk) the logit max m
//                  and the exp-sum l relative to it, and per (row, window) the
//                  window's exp-sum relative to the same m
//   k_obs_rows     per row: global max M and 1 / L from its chunks
//   k_obs_windows  per window: sum over KV heads and rows of
//                  l_window * exp(m - M) / L, divided by H_q
// Logits come from 16x16x32 bf16 MFMAs with the keys as the A operand (rows =
// 16 keys) and the query rows as the B operand (columns = 16 query rows): a
// lane holds 4 keys of one query row, so per-row sums fold in-lane and then
// over the lanes l, l ^ 16, l ^ 32, l ^ 48.  Each wave owns one chunk (its A operands
// stay in registers for every row); the query rows are staged in LDS, 128 at
// a time.
#include <mutex>

#include "qv_device.h"

namespace qv {

// Fixed scratch of the allocation-free entry point (qevict_prefill_scores_noalloc):
// every device the library runs on holds one copy for the life of the process.
// Host code never uses this name as an address: the per-device address comes
// from static_obs_scratch(), looked up once per device at cache creation.
static __device__ __align__(256) uint8_t scratch[kStaticObsScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// Device address of `scratch` on the current device (looked up on the first
// call for that device, with it current).  *what names the HIP call that failed.
hipError_t static_obs_scratch(void** ptr, const char** what) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *what = "hipGetDevice";
    return e;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    *what = "device index";
    return hipErrorInvalidDevice;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) {
      *what = "hipGetSymbolAddress";
      return e;
    }
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

constexpr int kObsChunkKeys = 64;      // keys per wave
constexpr int kObsRows = 128;          // query rows staged in LDS at once
constexpr int kObsRowBytes = 272;      // 256 B of a row + 16 B pad (conflict-free B reads)

__device__ __forceinline__ f32x4 mfma_obs(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// four workgroups per compute unit (at most 128 VGPRs); W8: 8-token windows (eight
// per chunk), a separate instantiation so the other window sizes carry none of it
template <bool W8>
__global__ __launch_bounds__(256, 4) void k_obs_chunks(ObsArgs a) {
  const int g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T, n_rows = a.n_rows;
  const int lr = lane & 15, lq = lane >> 4;
  const int c = blockIdx.x * 4 + wave;           // this wave's chunk
  const bool live = c < a.n_chunks;             // uniform per wave
  const int kbase = a.cbase + kObsChunkKeys * c;
  __shared__ __attribute__((aligned(16))) uint8_t sq[kObsRows * kObsRowBytes];

  // A operands: tile kt, k-step kc covers channels 32 kc + 8 lq .. + 7 of key
  // kbase + 16 kt + lr
  const uint16_t* kb = a.k + ((int64_t)b * a.H_kv + g) * T * kHeadDim;
  u32x4 kop[4][4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    const int key = kbase + 16 * kt + lr;
    const bool ok = live && key >= 0 && key < T;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
      kop[kt][kc] = ok ? *(const u32x4*)(kb + (int64_t)key * kHeadDim + 32 * kc + 8 * lq)
                       : (u32x4){0, 0, 0, 0};
  }
  const uint16_t* qb = a.q + ((int64_t)b * a.H_q + (int64_t)g * a.gqa) * a.n_obs * kHeadDim;
  const int pos0 = T - a.n_obs;   // position of observation row j = pos0 + j
  // only a chunk reaching below key 0 or past the first observation position masks keys
  const bool edge = kbase < 0 || kbase + kObsChunkKeys - 1 > pos0;
  const int wpc = kObsChunkKeys / a.W;          // windows per chunk: 8 (W = 8), 2 (W = 32) or 1 (W = 64)
  const int w0 = (c - a.n_pre) * wpc;           // first window of the chunk (< 0: sink chunk)
  const int64_t bg = (int64_t)b * a.H_kv + g;
  const float sc = a.scale_log2;
  // outputs of this chunk (uniform pointers): statistics, and the sums of its windows
  float2* const cml_out = a.cml + (bg * a.n_chunks + c) * n_rows;
  float* const wl_a = a.wl + (bg * a.n_w + w0) * n_rows;
  const bool has_a = w0 >= 0 && w0 < a.n_w;
  const bool has_b = wpc == 2 && w0 >= 0 && w0 + 1 < a.n_w;

  for (int r0 = 0; r0 < n_rows; r0 += kObsRows) {
    const int nr = min(kObsRows, n_rows - r0);
    __syncthreads();   // the previous rows are consumed
#pragma unroll 2
    for (int i = 0; i < kObsRows * 16 / 256; ++i) {
      const int e = tid + 256 * i, row = e >> 4, part = e & 15;
      const u32x4 v = row < nr ? *(const u32x4*)(qb + (int64_t)(r0 + row) * kHeadDim + 8 * part)
                               : (u32x4){0, 0, 0, 0};
      *(u32x4*)(sq + row * kObsRowBytes + 16 * part) = v;
    }
    __syncthreads();
    if (!live) continue;
    for (int rt = 0; rt < (nr + 15) / 16; ++rt) {
      const int row = rt * 16 + lr;   // this lane's query row inside the staged rows
      const int rg = r0 + row;
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
      // acc[kt][i]: raw logit of key kbase + 16 kt + 4 lq + i for this row
      if (edge) {
        const int pos = pos0 + (rg % a.n_obs);   // this row's query position
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = kbase + 16 * kt + 4 * lq + i;
            if (key < 0 || key > pos) acc[kt][i] = -INFINITY;
          }
      }
      float mr = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) mr = fmaxf(mr, acc[kt][i]);
      mr = rows_max(mr);
      const float m = mr * sc;                      // the chunk's max for this row, log2 units
      const float mu = mr > -INFINITY ? m : 0.f;    // all keys masked: every term is exp2(-inf) = 0
      float lA = 0.f, lB = 0.f;                     // keys of tiles 0-1 and 2-3
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        lA += __builtin_amdgcn_exp2f(fmaf(acc[0][i], sc, -mu));
        lA += __builtin_amdgcn_exp2f(fmaf(acc[1][i], sc, -mu));
        lB += __builtin_amdgcn_exp2f(fmaf(acc[2][i], sc, -mu));
        lB += __builtin_amdgcn_exp2f(fmaf(acc[3][i], sc, -mu));
      }
      if constexpr (W8) {
        // 8-token windows: tile kt holds windows 2 kt (lanes lq 0, 1) and 2 kt + 1
        // (lq 2, 3); the pair sums land in lanes lq 0 and 2
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          float lt = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) lt += __builtin_amdgcn_exp2f(fmaf(acc[kt][i], sc, -mu));
          lt += __shfl_xor(lt, 16, 64);
          const int w = w0 + 2 * kt + (lq >> 1);
          if (row < nr && (lq & 1) == 0 && w >= 0 && w < a.n_w) wl_a[(int64_t)(w - w0) * n_rows + rg] = lt;
        }
      }
      lA = rows_sum(lA);
      lB = rows_sum(lB);
      if (row < nr) {
        if (lq == 0) cml_out[rg] = make_float2(m, lA + lB);
        if constexpr (!W8) {
          if (lq == 1 && has_a) wl_a[rg] = wpc == 2 ? lA : lA + lB;
          if (lq == 2 && has_b) wl_a[n_rows + rg] = lB;
        }
      }
    }
  }
}

// (M, 1 / L) of every row from its chunks' (max, exp-sum) pairs: 256 / P rows
// per workgroup, thread (p, r) takes chunks p, p + P, ... of row r (consecutive
// threads read consecutive rows): first their max, then their sum relative to
// it; the P partial results of a row are folded by a pairwise tree (a fixed order).
// P = 16: 16 consecutive rows per workgroup keep the loads of a chunk's
// statistics in whole 128-byte lines (4 rows per workgroup read 32-byte pieces
// and were three times slower at 1024 chunks).
__device__ __forceinline__ float2 ml_combine(float2 x, float2 y) {
  const float mm = fmaxf(x.x, y.x);
  float ls = 0.f;
  if (x.x > -INFINITY) ls += x.y * __builtin_amdgcn_exp2f(x.x - mm);
  if (y.x > -INFINITY) ls += y.y * __builtin_amdgcn_exp2f(y.x - mm);
  return make_float2(mm, ls);
}

template <int P>
__global__ __launch_bounds__(256) void k_obs_rows(ObsArgs a) {
  constexpr int RPB = 256 / P;   // rows per workgroup
  const int g = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int rl = tid % RPB, p = tid / RPB, r = blockIdx.x * RPB + rl;
  const int64_t bg = (int64_t)b * a.H_kv + g;
  __shared__ float2 part[P][RPB];
  float m = -INFINITY, l = 0.f;
  if (r < a.n_rows) {
    const float2* cm = a.cml + bg * a.n_chunks * a.n_rows + r;
#pragma unroll 4
    for (int c = p; c < a.n_chunks; c += P) m = fmaxf(m, cm[(int64_t)c * a.n_rows].x);
    if (m > -INFINITY) {
#pragma unroll 4
      for (int c = p; c < a.n_chunks; c += P) {
        const float2 s = cm[(int64_t)c * a.n_rows];
        l += s.y * __builtin_amdgcn_exp2f(s.x - m);   // exp2(-inf) = 0 for empty chunks
      }
    }
  }
  part[p][rl] = make_float2(m, l);
  __syncthreads();
  for (int h = P / 2; h > 0; h >>= 1) {
    if (p < h) part[p][rl] = ml_combine(part[p][rl], part[p + h][rl]);
    __syncthreads();
  }
  if (p == 0 && r < a.n_rows) {
    const float2 t = part[0][rl];
    a.row_ml[bg * a.n_rows + r] = make_float2(t.x, t.y > 0.f ? 1.f / t.y : 0.f);
  }
}

// score[b][w] = (1 / H_q) * sum over KV heads and rows of l_w * exp2(m_c - M) / L.
// A workgroup of 256 threads serves wpw windows (1, 2 or 4: enough workgroups
// for the chip whatever the window count), 256 / wpw threads each: thread t of
// a window takes rows t, t + 256 / wpw, ... of every KV head; the window's sum
// is folded by a butterfly per wave, then its waves in order.
__global__ __launch_bounds__(256) void k_obs_windows(ObsArgs a, int wpw) {
  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tpw = 256 / wpw;                      // threads per window
  const int w = blockIdx.x * wpw + tid / tpw, t = tid % tpw;
  __shared__ float red[4];
  float s = 0.f;
  if (w < a.n_w) {
    const int c = a.n_pre + w / (kObsChunkKeys / a.W);
    // entries (g, r) = t, t + tpw, ... of the KV head x row list, stepped without division
    const int nr = a.n_rows, dg = tpw / nr, dr = tpw % nr;
    int g = t / nr, r = t % nr;
#pragma unroll 4
    while (g < a.H_kv) {
      const int64_t bg = (int64_t)b * a.H_kv + g;
      // M is finite for every row; a chunk with no visible key has m = -inf and l = 0
      const float2 rm = a.row_ml[bg * nr + r];
      const float m = a.cml[(bg * a.n_chunks + c) * nr + r].x;
      s += a.wl[(bg * a.n_w + w) * nr + r] * __builtin_amdgcn_exp2f(m - rm.x) * rm.y;
      r += dr;
      g += dg;
      if (r >= nr) {
        r -= nr;
        ++g;
      }
    }
  }
  for (int o = 1; o < 64; o <<= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) red[wave] = s;
  __syncthreads();
  const int wpwv = tpw / 64;                      // waves per window
  if (t == 0 && w < a.n_w) {
    const int w0 = wave;                          // this window's first wave
    float v = red[w0];
    for (int k = 1; k < wpwv; ++k) v += red[w0 + k];
    a.scores[(int64_t)b * a.n_w + w] = v / (float)a.H_q;
  }
}

hipError_t launch_prefill_scores(const ObsArgs& a, hipStream_t st) {
  if (a.n_w <= 0) return hipSuccess;
  if (a.W == 8) hipLaunchKernelGGL(k_obs_chunks<true>, dim3(a.n_blk, a.H_kv, a.B), dim3(256), 0, st, a);
  else hipLaunchKernelGGL(k_obs_chunks<false>, dim3(a.n_blk, a.H_kv, a.B), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_obs_rows<16>, dim3((a.n_rows + 15) / 16, a.H_kv, a.B), dim3(256), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t nwin = (int64_t)a.n_w * a.B;
  const int wpw = nwin >= 4096 ? 4 : nwin >= 2048 ? 2 : 1;   // windows per workgroup
  hipLaunchKernelGGL(k_obs_windows, dim3((a.n_w + wpw - 1) / wpw, a.B), dim3(256), 0, st, a, wpw);
  return hipGetLastError();
}

}  // namespace qv
