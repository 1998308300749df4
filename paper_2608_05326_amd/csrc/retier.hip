// Routing event: re-rank the candidate windows and re-tier them
// (QEvict Sec. 4.3 candidate pool and TopK equations; Algorithm 1).
//
// One 1024-thread workgroup per sequence:
//   1. candidates = current Full and Quantized windows (the live list, in
//      window order) followed by the windows that left the recent region;
//   2. 64-bit keys (score descending, then window ascending) define the total
//      order; the keys at positions K_f, K_f + ceil(K_q / 2) and K_f + K_q are
//      found by selection (histogram refinement), so no full sort is needed;
//   3. position < K_f -> Full, < K_f + K_q -> Quantized, else Evicted (the
//      one-way policy, Full only from candidates that are not Quantized,
//      sorts the keys and counts along the sorted order);
//   4. Algorithm 1 transitions: promotions keep the ledger dormant, first
//      demotions request a quantization, dormant ledgers are reactivated,
//      evictions release slots and delete the ledger;
//   5. freed slots are handed to the new requests in ascending slot order by
//      prefix sums (deterministic), and the quantize / promote work lists and
//      the new live list (window order, with split-balancing cost prefix) are
//      written for the kernels that follow on the stream.
#include "qv_device.h"

namespace qv {

// Total order key: ascending key = descending score, ties to the lower candidate
// index (candidates are stored in window order, so this is the lower window).
__device__ __forceinline__ uint64_t rank_key(float f, uint32_t cand) {
  if (f == 0.f) f = 0.f;   // -0 and +0 compare equal
  const uint32_t u = __float_as_uint(f);
  const uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)(~asc) << 32) | cand;
}

// Inclusive prefix sum over the 64 lanes of a wave: row shifts 1, 2, 4, 8 within
// 16-lane rows, then row broadcasts of lanes 15 and 31 (DPP, no LDS traffic).
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);   // row_bcast:15 -> rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);   // row_bcast:31 -> rows 2, 3
  return x;
}

// Exclusive prefix sums of NV arrays at once (each buf[v][0..n[v]), n <= kMaxCand),
// in place; tot[v] receives each total.  One pair of barriers for all arrays.
template <int NV>
__device__ __forceinline__ void block_scan_multi(int32_t* const (&buf)[NV], const int (&n)[NV], int (&tot)[NV],
                                 int32_t* tmp /* >= NV * 16 */) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int PER = kMaxCand / kRetierThreads;
  constexpr int NW = kRetierThreads / 64;
  int v[NV][PER], sum[NV], x[NV];
#pragma unroll
  for (int a = 0; a < NV; ++a) {
    sum[a] = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = tid * PER + k;
      v[a][k] = i < n[a] ? buf[a][i] : 0;
      sum[a] += v[a][k];
    }
    x[a] = wave_inclusive_scan(sum[a]);
    if (lane == 63) tmp[a * NW + wave] = x[a];
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < NV; ++a) {
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const int t = tmp[a * NW + w];
      before += w < wave ? t : 0;
      total += t;
    }
    tot[a] = total;
    int run = x[a] - sum[a] + before;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = tid * PER + k;
      if (i < n[a]) buf[a][i] = run;
      run += v[a][k];
    }
  }
  __syncthreads();
}

// Exclusive prefix counts of NV flag arrays held in registers in strided
// layout (element c = tid + k * kRetierThreads, k < PER): rank[v][k] = set flags
// before element c, tot[v] = set flags in all.  Only slices k < kmax (uniform)
// may hold set flags; the others are skipped.  Wave ballots, then one wave per
// array scans the (slice, wave) counts; two barriers.
template <int NV>
__device__ __forceinline__ void flag_scan(const bool (&f)[NV][kMaxCand / kRetierThreads],
                                          int (&rank)[NV][kMaxCand / kRetierThreads], int (&tot)[NV],
                                          int32_t* tmp /* >= NV * 64 + NV */, int kmax) {
  constexpr int PER = kMaxCand / kRetierThreads;
  constexpr int NW = kRetierThreads / 64;
  static_assert(PER * NW == 64, "one wave scans the slice counts");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (k >= kmax) break;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const uint64_t bl = __builtin_amdgcn_ballot_w64(f[v][k]);
      rank[v][k] = __popcll(bl & below);
      if (lane == 0) tmp[v * 64 + k * NW + wave] = __popcll(bl);
    }
  }
  __syncthreads();
  if (wave < NV) {
    const int x = lane < kmax * NW ? tmp[wave * 64 + lane] : 0;
    const int inc = wave_inclusive_scan(x);
    tmp[wave * 64 + lane] = inc - x;
    if (lane == 63) tmp[NV * 64 + wave] = inc;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (k >= kmax) break;
#pragma unroll
    for (int v = 0; v < NV; ++v) rank[v][k] += tmp[v * 64 + k * NW + wave];
  }
#pragma unroll
  for (int v = 0; v < NV; ++v) tot[v] = tmp[NV * 64 + v];
}

// Value of `x` held by lane (lane ^ J), J in {1, 2, 4, 8, 16, 32}; VALU only.
template <int J>
__device__ __forceinline__ uint32_t lane_xor(uint32_t x, int lane) {
  if constexpr (J == 1) {
    return __builtin_amdgcn_update_dpp(0u, x, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
  } else if constexpr (J == 2) {
    return __builtin_amdgcn_update_dpp(0u, x, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
  } else if constexpr (J == 4) {
    const uint32_t dn = __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xF, 0xF, false);  // row_shr:4
    const uint32_t up = __builtin_amdgcn_update_dpp(0u, x, 0x104, 0xF, 0xF, false);  // row_shl:4
    return (lane & 4) ? dn : up;
  } else if constexpr (J == 8) {
    return __builtin_amdgcn_update_dpp(0u, x, 0x128, 0xF, 0xF, false);  // row_ror:8
  } else if constexpr (J == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    const uint32_t r0 = r[0], r1 = r[1];
    return (lane & 16) ? r0 : r1;
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    const uint32_t r0 = r[0], r1 = r[1];
    return (lane & 32) ? r0 : r1;
  }
}

// One compare-exchange stage (block size k, distance j) on positions t + m * NT.
template <int KP>
__device__ __forceinline__ void cmpx_stage(uint64_t (&key)[KP], const uint64_t (&other)[KP], int k,
                                           int j) {
#pragma unroll
  for (int m = 0; m < KP; ++m) {
    const int i = threadIdx.x + m * kRetierThreads;
    const bool up = (i & k) == 0, lower = (i & j) == 0;
    const uint64_t a = key[m], b = other[m];
    key[m] = (up == lower) ? (a < b ? a : b) : (a < b ? b : a);
  }
}

template <int J, int KP>
__device__ __forceinline__ void reg_stage(uint64_t (&key)[KP], int k, int lane) {
  uint64_t other[KP];
#pragma unroll
  for (int m = 0; m < KP; ++m) {
    const uint32_t lo = lane_xor<J>((uint32_t)key[m], lane);
    const uint32_t hi = lane_xor<J>((uint32_t)(key[m] >> 32), lane);
    other[m] = ((uint64_t)hi << 32) | lo;
  }
  cmpx_stage<KP>(key, other, k, J);
}

// Bitonic sort (ascending) of KP keys per thread; thread t holds positions
// t + m * kRetierThreads.  Partners closer than 64 positions are exchanged in
// registers (DPP / permlane), partners 64..1023 apart through LDS, farther ones
// inside a thread.
template <int KP>
__device__ void bitonic_sort(uint64_t (&key)[KP], int n_pow, uint64_t* lds) {
  const int t = threadIdx.x, lane = t & 63;
  // with one key per thread only the waves holding positions < n_pow take part
  const bool act = KP > 1 || (t >> 6) < ((n_pow + 63) >> 6);
  for (int k = 2; k <= n_pow; k <<= 1) {
    for (int j = k >> 1; j >= 64; j >>= 1) {
      if (j >= kRetierThreads) {
        const int mj = j / kRetierThreads;
#pragma unroll
        for (int m = 0; m < KP; ++m) {
          const int mp = m ^ mj;
          if (mp > m && mp < KP) {
            const int i = t + m * kRetierThreads;
            const bool up = (i & k) == 0;
            const uint64_t x = key[m], y = key[mp];
            if ((x > y) == up) { key[m] = y; key[mp] = x; }
          }
        }
      } else {
        uint64_t other[KP];
        if (act) {
#pragma unroll
          for (int m = 0; m < KP; ++m) lds[t + m * kRetierThreads] = key[m];
        }
        __syncthreads();
        if (act) {
#pragma unroll
          for (int m = 0; m < KP; ++m) other[m] = lds[(t + m * kRetierThreads) ^ j];
        }
        __syncthreads();
        if (act) cmpx_stage<KP>(key, other, k, j);
      }
    }
    if (act) {
      if (k > 32) reg_stage<32, KP>(key, k, lane);
      if (k > 16) reg_stage<16, KP>(key, k, lane);
      if (k > 8) reg_stage<8, KP>(key, k, lane);
      if (k > 4) reg_stage<4, KP>(key, k, lane);
      if (k > 2) reg_stage<2, KP>(key, k, lane);
      reg_stage<1, KP>(key, k, lane);
    }
  }
}

template <int KP>
__device__ void sort_candidates(uint64_t* skey, int n_cand, int n_pow) {
  uint64_t key[KP];
#pragma unroll
  for (int m = 0; m < KP; ++m) {
    const int i = threadIdx.x + m * kRetierThreads;
    key[m] = i < n_cand ? skey[i] : ~0ull;
  }
  __syncthreads();
  bitonic_sort<KP>(key, n_pow, skey);
#pragma unroll
  for (int m = 0; m < KP; ++m) skey[threadIdx.x + m * kRetierThreads] = key[m];
  __syncthreads();
}

// Exchange-compare within a wave (lane index as position, J < 64).
template <int J>
__device__ __forceinline__ uint64_t wave_cmpx(uint64_t x, int k, int lane) {
  const uint32_t lo = lane_xor<J>((uint32_t)x, lane);
  const uint32_t hi = lane_xor<J>((uint32_t)(x >> 32), lane);
  const uint64_t y = ((uint64_t)hi << 32) | lo;
  const bool up = (lane & k) == 0, lower = (lane & J) == 0;
  return (up == lower) ? (x < y ? x : y) : (x < y ? y : x);
}

// Ascending bitonic sort of one key per lane across a wave (lane exchanges only).
__device__ __forceinline__ uint64_t wave_sort64(uint64_t x, int lane) {
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1) {
    if (k >= 64) x = wave_cmpx<32>(x, k, lane);
    if (k >= 32) x = wave_cmpx<16>(x, k, lane);
    if (k >= 16) x = wave_cmpx<8>(x, k, lane);
    if (k >= 8) x = wave_cmpx<4>(x, k, lane);
    if (k >= 4) x = wave_cmpx<2>(x, k, lane);
    x = wave_cmpx<1>(x, k, lane);
  }
  return x;
}

// Sort of up to kRetierThreads unique keys: every wave sorts its run of 64 in
// registers, then a key's final position is its lane in its run plus, for each
// other run, the number of that run's keys below it (binary searches in LDS
// that advance together, NR = run count rounded up to a power of two).
template <int NR>
__device__ __forceinline__ int rank_in_runs(const uint64_t* skey, uint64_t x, int wave, int n_runs) {
  int lo[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) lo[r] = 0;
#pragma unroll
  for (int step = 64; step >= 1; step >>= 1) {
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const int idx = lo[r] + step - 1;
      const uint64_t v = skey[64 * r + (idx < 64 ? idx : 63)];
      lo[r] += (r < n_runs && r != wave && idx < 64 && v < x) ? step : 0;
    }
  }
  int rank = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) rank += lo[r];
  return rank;
}

__device__ void sort_runs(uint64_t* skey, int n_cand) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int n_runs = (n_cand + 63) >> 6;
  uint64_t x = t < n_cand ? skey[t] : ~0ull;
  __syncthreads();
  if (wave < n_runs) {
    x = wave_sort64(x, lane);
    skey[t] = x;
  }
  __syncthreads();
  int rank = lane;
  if (wave < n_runs) {
    if (n_runs <= 2) rank += rank_in_runs<2>(skey, x, wave, n_runs);
    else if (n_runs <= 4) rank += rank_in_runs<4>(skey, x, wave, n_runs);
    else if (n_runs <= 8) rank += rank_in_runs<8>(skey, x, wave, n_runs);
    else rank += rank_in_runs<16>(skey, x, wave, n_runs);
  }
  __syncthreads();
  if (wave < n_runs && x != ~0ull) skey[rank] = x;
  __syncthreads();
}

// Minimum and maximum of one 64-bit value per lane across a wave (VALU only).
template <int J>
__device__ __forceinline__ void minmax_step(uint64_t& mn, uint64_t& mx, int lane) {
  const uint64_t a = ((uint64_t)lane_xor<J>((uint32_t)(mn >> 32), lane) << 32) | lane_xor<J>((uint32_t)mn, lane);
  const uint64_t b = ((uint64_t)lane_xor<J>((uint32_t)(mx >> 32), lane) << 32) | lane_xor<J>((uint32_t)mx, lane);
  mn = a < mn ? a : mn;
  mx = b > mx ? b : mx;
}

// Order statistics of the candidate keys (unique 64-bit values, thread t holding
// candidates t + k * kRetierThreads, k < kc, c < n_cand): thr[i] = the key at
// ascending position target[i], or ~0 when target[i] >= n_cand or the target is
// not asked for (want bit i clear).  Sorted position p < target[i] then holds
// exactly for the keys below thr[i].
//
// Each target keeps a key interval [lo, hi] that contains its key and the rank
// r of that key within the interval.  A round splits an interval of span 2^m
// into at most 1024 equal buckets (width 2^(m-10)), counts the keys per bucket
// and keeps the bucket holding rank r: ten bits of the interval per round, so
// at most seven rounds for 64-bit keys, and one round when the first split
// already leaves at most kSelSmall keys in the bucket (the usual case).  The
// keys of the final interval (at most kSelSmall) are then ranked by pairwise
// comparison.  LDS: `hist` 3 x 1024 counters, `sel` the intervals and results.
constexpr int kSelBuckets = 1024;
constexpr int kSelSmall = 64;
struct SelLds {
  int32_t hist[3][kSelBuckets];
  uint64_t list[3][kSelSmall];
  uint64_t wmin[kRetierThreads / 64], wmax[kRetierThreads / 64];
  uint64_t lo[3], hi[3], thr[3];
  int32_t r[3], cnt[3], nlist[3];
  // one-round path (select_tiers)
  uint32_t swmin[kRetierThreads / 64], swmax[kRetierThreads / 64];
  uint32_t blo[3], bhi[3];
  int32_t br[3], bcnt[3];
};

__device__ void select_thresholds(const uint64_t (&key)[kMaxCand / kRetierThreads], int kc, int n_cand,
                                  const int (&target)[3], int want, SelLds& s, uint64_t (&thr)[3]) {
  constexpr int PER = kMaxCand / kRetierThreads;
  constexpr int NW = kRetierThreads / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 3 * kSelBuckets; i += kRetierThreads) (&s.hist[0][0])[i] = 0;
  if (tid < 3) s.nlist[tid] = 0;
  uint64_t mn = ~0ull, mx = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (k < kc && tid + k * kRetierThreads < n_cand) {
      mn = key[k] < mn ? key[k] : mn;
      mx = key[k] > mx ? key[k] : mx;
    }
  }
  minmax_step<1>(mn, mx, lane);
  minmax_step<2>(mn, mx, lane);
  minmax_step<4>(mn, mx, lane);
  minmax_step<8>(mn, mx, lane);
  minmax_step<16>(mn, mx, lane);
  minmax_step<32>(mn, mx, lane);
  if (lane == 0) {
    s.wmin[wave] = mn;
    s.wmax[wave] = mx;
  }
  __syncthreads();
  mn = ~0ull;
  mx = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    mn = s.wmin[w] < mn ? s.wmin[w] : mn;
    mx = s.wmax[w] > mx ? s.wmax[w] : mx;
  }
  uint64_t lo[3], hi[3];
  int r[3], cnt[3];
  bool act[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    act[i] = ((want >> i) & 1) != 0 && target[i] >= 0 && target[i] < n_cand;
    lo[i] = mn;
    hi[i] = mx;
    r[i] = target[i];
    cnt[i] = n_cand;
  }
  // uniform across the workgroup: every thread holds the same intervals
  for (int round = 0; round < 8; ++round) {
    bool refine[3];
    int sh[3];
    bool any = false;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      refine[i] = act[i] && cnt[i] > kSelSmall;
      const uint64_t span = hi[i] - lo[i];
      const int bl = span == 0 ? 0 : 64 - __builtin_clzll(span);
      sh[i] = bl > 10 ? bl - 10 : 0;
      any |= refine[i];
    }
    if (!any) break;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (k >= kc || tid + k * kRetierThreads >= n_cand) continue;
      const uint64_t x = key[k];
#pragma unroll
      for (int i = 0; i < 3; ++i)
        if (refine[i] && x >= lo[i] && x <= hi[i]) atomicAdd(&s.hist[i][(int)((x - lo[i]) >> sh[i])], 1);
    }
    __syncthreads();
    // wave i scans target i's counters (16 per lane), clears them for the next
    // round and publishes the bucket that holds rank r
    if (wave < 3 && refine[wave]) {
      const int i = wave;
      int h[16];
      int4* row = (int4*)&s.hist[i][16 * lane];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int4 v = row[q];
        h[4 * q] = v.x; h[4 * q + 1] = v.y; h[4 * q + 2] = v.z; h[4 * q + 3] = v.w;
        row[q] = make_int4(0, 0, 0, 0);
      }
      int sum = 0;
#pragma unroll
      for (int j = 0; j < 16; ++j) sum += h[j];
      const int inc = wave_inclusive_scan(sum);
      const int exc = inc - sum;
      if (exc <= r[i] && r[i] < inc) {   // exactly one lane
        int cum = exc, bk = 0, nr = 0, nc = 0;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          if (nc == 0 && r[i] < cum + h[j]) {
            bk = 16 * lane + j;
            nr = r[i] - cum;
            nc = h[j];
          }
          cum += h[j];
        }
        const uint64_t nlo = lo[i] + ((uint64_t)bk << sh[i]);
        const uint64_t wd = (1ull << sh[i]) - 1;
        const uint64_t top = nlo > ~0ull - wd ? ~0ull : nlo + wd;
        s.lo[i] = nlo;
        s.hi[i] = top < hi[i] ? top : hi[i];
        s.r[i] = nr;
        s.cnt[i] = nc;
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      if (refine[i]) {
        lo[i] = s.lo[i];
        hi[i] = s.hi[i];
        r[i] = s.r[i];
        cnt[i] = s.cnt[i];
      }
    }
  }
  // the keys left in each interval, ranked pairwise
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (k >= kc || tid + k * kRetierThreads >= n_cand) continue;
    const uint64_t x = key[k];
#pragma unroll
    for (int i = 0; i < 3; ++i)
      if (act[i] && x >= lo[i] && x <= hi[i]) {
        const int p = atomicAdd(&s.nlist[i], 1);
        if (p < kSelSmall) s.list[i][p] = x;
      }
  }
  __syncthreads();
  if (wave < 3 && act[wave]) {
    const int i = wave;
    const int n = cnt[i];
    const uint64_t x = lane < n ? s.list[i][lane] : ~0ull;
    int below = 0;
    for (int j = 0; j < n; ++j) below += s.list[i][j] < x ? 1 : 0;
    if (lane < n && below == r[i]) s.thr[i] = x;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 3; ++i) thr[i] = act[i] ? s.thr[i] : ~0ull;
}

// Upper word of a candidate's key: the score part (a monotone map of the float)
__device__ __forceinline__ uint32_t key_hi(float f) { return (uint32_t)(rank_key(f, 0u) >> 32); }

// Minimum and maximum of one 32-bit value per lane across a wave, valid in lane
// 63 (row shifts within 16-lane rows, then row broadcasts; DPP, no LDS).
__device__ __forceinline__ void wave_minmax_u32(uint32_t& mn, uint32_t& mx) {
#define QV_MM(ctrl, rmask)                                                                   \
  mn = min(mn, (uint32_t)__builtin_amdgcn_update_dpp((int)mn, (int)mn, ctrl, rmask, 0xF, false)); \
  mx = max(mx, (uint32_t)__builtin_amdgcn_update_dpp((int)mx, (int)mx, ctrl, rmask, 0xF, false));
  QV_MM(0x111, 0xF)   // row_shr:1
  QV_MM(0x112, 0xF)   // row_shr:2
  QV_MM(0x114, 0xF)   // row_shr:4
  QV_MM(0x118, 0xF)   // row_shr:8
  QV_MM(0x142, 0xA)   // row_bcast:15 -> rows 1, 3
  QV_MM(0x143, 0xC)   // row_bcast:31 -> rows 2, 3
#undef QV_MM
}

// Tier positions of the candidates in one histogram round (the usual case).
// Before this call (ahead of the barrier that follows the first loads) every
// wave has stored the minimum and maximum upper key word of its candidates in
// s.swmin / s.swmax, and s.hist[0] and s.nlist are zero.  The range of upper
// words is cut into at most 1024 equal buckets; for each target the bucket that
// holds its position, the rank r within it and its count are found.  A key
// below the bucket lies below the target; a key above it does not; a key in a
// bucket of one key is the target's own key; in a bucket of more keys its rank
// among them is compared with r.  A bucket of more than kSelSmall keys (ties or
// heavy clustering) falls back to the general refinement (select_thresholds).
// Result: bit i of below[k] is set when key k lies below position target[i]
// (always set for a target past the last candidate or not asked for).
__device__ void select_tiers(const uint64_t (&key)[kMaxCand / kRetierThreads], int kc, int n_cand,
                             const int (&target)[3], int want, SelLds& s,
                             uint32_t (&below)[kMaxCand / kRetierThreads]) {
  constexpr int PER = kMaxCand / kRetierThreads;
  constexpr int NW = kRetierThreads / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  bool act[3];
  bool any = false;
  uint32_t all = 0;
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    act[i] = ((want >> i) & 1) != 0 && target[i] >= 0 && target[i] < n_cand;
    any |= act[i];
    all |= act[i] ? 0u : 1u << i;
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) below[k] = all;
  if (!any) return;
  uint32_t mn = ~0u, mx = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    mn = min(mn, s.swmin[w]);
    mx = max(mx, s.swmax[w]);
  }
  mn = __builtin_amdgcn_readfirstlane(mn);
  mx = __builtin_amdgcn_readfirstlane(mx);
  const uint32_t span = mx - mn;
  const int bl = span == 0 ? 0 : 32 - __builtin_clz(span);
  const int sh = bl > 10 ? bl - 10 : 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (k >= kc || tid + k * kRetierThreads >= n_cand) continue;
    atomicAdd(&s.hist[0][((uint32_t)(key[k] >> 32) - mn) >> sh], 1);
  }
  __syncthreads();
  // wave i finds target i's bucket (16 counters per lane)
  if (wave < 3 && act[wave]) {
    const int i = wave;
    const int t = target[i];
    int h[16];
    const int4* row = (const int4*)&s.hist[0][16 * lane];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int4 v = row[q];
      h[4 * q] = v.x; h[4 * q + 1] = v.y; h[4 * q + 2] = v.z; h[4 * q + 3] = v.w;
    }
    int sum = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) sum += h[j];
    const int inc = wave_inclusive_scan(sum);
    const int exc = inc - sum;
    if (exc <= t && t < inc) {   // exactly one lane
      // bucket j of this lane: the first whose running end passes t
      int cum = exc, bk = 0, before = exc, nc = 0;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const bool past = cum + h[j] <= t;
        bk += past ? 1 : 0;
        before = past ? cum + h[j] : before;
        cum += h[j];
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) nc = j == bk ? h[j] : nc;
      const uint32_t b = (uint32_t)(16 * lane + bk);
      const uint64_t top = ((uint64_t)b << sh) + ((1ull << sh) - 1);
      s.blo[i] = mn + (b << sh);
      s.bhi[i] = mn + (uint32_t)(top < span ? top : span);
      s.br[i] = t - before;
      s.bcnt[i] = nc;
    }
  }
  __syncthreads();
  uint64_t lo[3], hi[3];
  int r[3], cnt[3];
  bool big = false, need_list = false;
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    lo[i] = (uint64_t)__builtin_amdgcn_readfirstlane(s.blo[i]) << 32;
    hi[i] = ((uint64_t)__builtin_amdgcn_readfirstlane(s.bhi[i]) << 32) | 0xFFFFFFFFull;
    r[i] = __builtin_amdgcn_readfirstlane(s.br[i]);
    cnt[i] = __builtin_amdgcn_readfirstlane(s.bcnt[i]);
    big |= act[i] && cnt[i] > kSelSmall;
    need_list |= act[i] && cnt[i] > 1;
  }
  if (big) {
    uint64_t thr[3];
    select_thresholds(key, kc, n_cand, target, want, s, thr);
#pragma unroll
    for (int k = 0; k < PER; ++k)
      below[k] = (key[k] < thr[0] ? 1u : 0u) | (key[k] < thr[1] ? 2u : 0u) | (key[k] < thr[2] ? 4u : 0u);
    return;
  }
  if (need_list) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (k >= kc || tid + k * kRetierThreads >= n_cand) continue;
      const uint64_t x = key[k];
#pragma unroll
      for (int i = 0; i < 3; ++i)
        if (act[i] && cnt[i] > 1 && x >= lo[i] && x <= hi[i]) {
          const int p = atomicAdd(&s.nlist[i], 1);
          if (p < kSelSmall) s.list[i][p] = x;
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (k >= kc || tid + k * kRetierThreads >= n_cand) continue;
    const uint64_t x = key[k];
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      bool b = true;
      if (act[i]) {
        if (x < lo[i]) {
          b = true;
        } else if (x > hi[i] || cnt[i] <= 1) {
          b = false;   // above the bucket, or the target's own key
        } else {
          int rk = 0;
          for (int j = 0; j < cnt[i]; ++j) rk += s.list[i][j] < x ? 1 : 0;
          b = rk < r[i];
        }
      }
      m |= b ? 1u << i : 0u;
    }
    below[k] = m;
  }
}

__global__ __launch_bounds__(kRetierThreads) void k_retier(RetierArgs a) {
  const Geometry& G = a.g;
  const int b = blockIdx.x, tid = threadIdx.x;
  const RetierUnit& U = a.unit[blockIdx.y];   // this workgroup's layer
  constexpr int NT = kRetierThreads;
  constexpr int PER = kMaxCand / NT;

  __shared__ __attribute__((aligned(16))) uint64_t skey[kMaxCand];   // sort keys or SelLds
  __shared__ int32_t sinfo[kMaxCand];
  __shared__ int32_t sa[kMaxCand];
  __shared__ int32_t sown[2 * kMaxCand];      // slot owners: Full slots, then quantized slots
  __shared__ int32_t tmp[5 * 64 + 16];
  __shared__ int32_t sstat[ST_N];
  int32_t* sb = (int32_t*)skey;               // after the sort: two more int arrays
  int32_t* fown = sown;
  int32_t* qown = sown + G.n_fslots;

  uint8_t* ub = U.base + (int64_t)b * a.L.unit_bytes;
  int8_t* tier = (int8_t*)(ub + a.L.tier);
  int8_t* ledger = (int8_t*)(ub + a.L.ledger);
  int8_t* bits = (int8_t*)(ub + a.L.bits);
  int32_t* fslot = (int32_t*)(ub + a.L.fslot);
  int32_t* qslot = (int32_t*)(ub + a.L.qslot);
  float* score = (float*)(ub + a.L.score);
  int32_t* fowner = (int32_t*)(ub + a.L.fowner);
  int32_t* qowner = (int32_t*)(ub + a.L.qowner);
  int32_t* iwin = (int32_t*)(ub + a.L.item_win);
  int32_t* iref = (int32_t*)(ub + a.L.item_ref);
  int32_t* icost = (int32_t*)(ub + a.L.item_cost);
  int32_t* iaux = (int32_t*)(ub + a.L.item_aux);
  float* iscore = (float*)(ub + a.L.item_score);
  int32_t* qlist = (int32_t*)(ub + a.L.qlist);
  int32_t* plist = (int32_t*)(ub + a.L.plist);
  int32_t* counts = (int32_t*)(ub + a.L.counts);
  int32_t* stats = (int32_t*)(ub + a.L.stats);

  // a routing batch whose wait for the cache stream timed out leaves the layer as it
  // is: the word is read with the first round of loads and tested before any store
  const int gate_failed =
      a.gate_fail ? __hip_atomic_load(a.gate_fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
  if (tid < ST_N) sstat[tid] = 0;
  // ---- one round of loads: the live list carries every candidate's state.
  // Entries are read up to the list's capacity without waiting for its length;
  // the slot owner tables and the scores of the windows entering the pool (a
  // range known from the arguments) are read in the same round.
  const int n_aged = U.aged_w1 - U.aged_w0;
  const int ko = (max(G.n_fslots, G.n_qslots) + NT - 1) / NT;   // owner-table slices
  int spec_ref[PER], spec_aux[PER], spec_win[PER], spec_fo[PER], spec_qo[PER];
  float spec_sc[PER], spec_aged[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = tid + k * NT;
    const bool ok = !a.prefill && c < G.max_fq;
    spec_ref[k] = ok ? iref[c] : 0;
    spec_aux[k] = ok ? iaux[c] : -1;
    spec_win[k] = ok ? iwin[c] : -1;
    spec_sc[k] = ok ? iscore[c] : 0.f;
    spec_fo[k] = k < ko && c < G.n_fslots ? fowner[c] : -1;
    spec_qo[k] = k < ko && c < G.n_qslots ? qowner[c] : -1;
    const int w = U.aged_w0 + c;
    spec_aged[k] = c >= n_aged ? 0.f
                 : (a.prefill ? a.init_scores[(int64_t)b * a.n_init + w] : score[w]);
  }
  // scores of the windows that follow the routed range (the next steps' recent
  // region; at most NR of them have started)
  float ring_sc = 0.f;
  if (tid < G.NR) {
    const int w = U.aged_w1 + tid;
    if (a.prefill) ring_sc = w < a.n_init ? a.init_scores[(int64_t)b * a.n_init + w] : 0.f;
    else ring_sc = w < G.nwc ? score[w] : 0.f;
  }
  const int n_fq = a.prefill ? 0 : counts[CNT_ITEMS];
  const int n_cand = n_fq + n_aged;
  if (gate_failed) {
    if (tid == 0) set_error(counts, ERR_GATE);
    return;
  }
  if (n_cand > kMaxCand) {
    if (tid == 0) set_error(counts, ERR_CAND);
    return;
  }
  const int kc = (n_cand + NT - 1) / NT;   // candidate slices in use
  // owner tables and entering scores to LDS (sinfo is free until tiering)
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = tid + k * NT;
    if (k < ko) {
      if (c < G.n_fslots) fown[c] = spec_fo[k];
      if (c < G.n_qslots) qown[c] = spec_qo[k];
    }
    if (c < n_aged) sinfo[c] = __float_as_int(spec_aged[k]);
  }
  if (a.prefill) {   // every prompt window (partial ones too) starts at its initial score
    for (int w = tid; w < a.n_init; w += NT) {
      const float v = a.init_scores[(int64_t)b * a.n_init + w];
      if (!__builtin_isfinite(v)) set_error(counts, ERR_NONFINITE);
      score[w] = v;
    }
  }
  // tier selection, ahead of the barrier: the range of the candidates' upper key
  // words per wave, and cleared first-round counters
  const bool one_way = (G.flags & 1u) != 0;
  SelLds& sel = *reinterpret_cast<SelLds*>(skey);
  if (!one_way) {
    const int lane = tid & 63, wave = tid >> 6;
    uint32_t wlo = ~0u, whi = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int c = tid + k * NT;
      if (c < n_fq) {
        const uint32_t u = key_hi(spec_sc[k]);
        wlo = min(wlo, u);
        whi = max(whi, u);
      }
      if (c < n_aged) {
        const uint32_t u = key_hi(spec_aged[k]);
        wlo = min(wlo, u);
        whi = max(whi, u);
      }
    }
    wave_minmax_u32(wlo, whi);
    if (lane == 63) {
      sel.swmin[wave] = wlo;
      sel.swmax[wave] = whi;
    }
    for (int i = tid; i < kSelBuckets; i += NT) sel.hist[0][i] = 0;
    if (tid < 3) sel.nlist[tid] = 0;
  }
  __syncthreads();

  int my_w[PER], my_old[PER], my_led[PER], my_fs[PER], my_qs[PER], my_bits[PER];
  float my_sc[PER];
  uint64_t my_key[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = tid + k * NT;
    my_w[k] = -1;
    my_sc[k] = 0.f;
    my_key[k] = ~0ull;
    if (k >= kc || c >= n_cand) continue;
    if (c < n_fq) {
      const int32_t ref = spec_ref[k], aux = spec_aux[k];
      const int kind = ref >> 28, slot = ref & 0x0FFFFFFF;
      my_w[k] = spec_win[k];
      my_sc[k] = spec_sc[k];
      if (kind == KIND_BF16) {
        my_old[k] = T_FULL;
        my_fs[k] = slot;
        my_qs[k] = aux < 0 ? -1 : (aux & 0x0FFFFFFF);
        my_led[k] = aux < 0 ? L_NONE : L_DORMANT;
        my_bits[k] = aux < 0 ? 0 : (aux >> 28);
      } else {
        my_old[k] = T_QUANT;
        my_fs[k] = -1;
        my_qs[k] = slot;
        my_led[k] = L_ACTIVE;
        my_bits[k] = kind == KIND_Q4 ? 4 : 2;
      }
    } else {
      my_w[k] = U.aged_w0 + (c - n_fq);
      my_sc[k] = __int_as_float(sinfo[c - n_fq]);
      my_old[k] = T_OPEN;   // aged, entering the pool
      my_fs[k] = -1;
      my_qs[k] = -1;
      my_led[k] = L_NONE;
      my_bits[k] = 0;
    }
    if (!__builtin_isfinite(my_sc[k])) set_error(counts, ERR_NONFINITE);
    my_key[k] = rank_key(my_sc[k], (uint32_t)c);
    if (one_way) skey[c] = my_key[k];
  }

  // ---- tier by sorted position ----
  // info = new tier | (position - K_f) << 8; only whether that rank lies in the
  // upper half of the Quantized tier is used (mixed widths)
  const int half_q = (G.K_q + 1) / 2;
  int my_info[PER];
  if (!one_way) {
    // the three positions that decide a tier and a width, found by selection
    // (no full sort): p < K_f <=> key < thr[0], p < K_f + half_q <=> key < thr[1],
    // p < K_f + K_q <=> key < thr[2]
    const int target[3] = {G.K_f, G.K_f + half_q, G.K_f + G.K_q};
    uint32_t bel[PER];
    select_tiers(my_key, kc, n_cand, target, G.bits_cfg == 42 ? 7 : 5, sel, bel);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int nt = (bel[k] & 1u) ? T_FULL : ((bel[k] & 4u) ? T_QUANT : T_EVICTED);
      my_info[k] = nt | (((bel[k] & 2u) ? 0 : half_q) << 8);
    }
  } else {
    int n_pow = 1;
    while (n_pow < n_cand) n_pow <<= 1;
    __syncthreads();
    if (n_cand <= NT) sort_runs(skey, n_cand);
    else if (n_pow <= NT) sort_candidates<1>(skey, n_cand, n_pow);
    else if (n_pow <= 2 * NT) sort_candidates<2>(skey, n_cand, n_pow);
    else sort_candidates<4>(skey, n_cand, n_pow);
    // Full only from candidates that are not currently Quantized
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int c = tid + k * NT;
      if (c < n_cand) sinfo[c] = my_old[k];
    }
    __syncthreads();
    for (int p = tid; p < n_cand; p += NT) {
      const int c = (int)(skey[p] & 0xFFFFFFFFu);
      sa[p] = sinfo[c] != T_QUANT ? 1 : 0;
    }
    __syncthreads();
    {
      int32_t* const bufs[1] = {sa};
      const int ns[1] = {n_cand};
      int tots[1];
      block_scan_multi<1>(bufs, ns, tots, tmp);
    }
    for (int p = tid; p < n_cand; p += NT) {
      const int c = (int)(skey[p] & 0xFFFFFFFFu);
      const bool f = sinfo[c] != T_QUANT && sa[p] < G.K_f;
      sa[p] = f ? 0 : 1;
      sinfo[c] = f ? T_FULL : 0;
    }
    __syncthreads();
    {
      int32_t* const bufs[1] = {sa};
      const int ns[1] = {n_cand};
      int tots[1];
      block_scan_multi<1>(bufs, ns, tots, tmp);
    }
    for (int p = tid; p < n_cand; p += NT) {
      const int c = (int)(skey[p] & 0xFFFFFFFFu);
      if (sinfo[c] != T_FULL) {
        const int rq = sa[p];
        sinfo[c] = (rq < G.K_q ? T_QUANT : T_EVICTED) | (rq << 8);
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int c = tid + k * NT;
      my_info[k] = k < kc && c < n_cand ? sinfo[c] : T_EVICTED;
    }
  }

  // ---- transitions; release slots (in the LDS owner tables) ----
  int my_nt[PER], my_req[PER], my_nb[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = tid + k * NT;
    my_req[k] = 0;
    my_nt[k] = T_EVICTED;
    if (k >= kc || c >= n_cand) continue;
    const int info = my_info[k];
    const int nt = info & 0xFF, rq = info >> 8;
    const int old = my_old[k], led = my_led[k];
    my_nt[k] = nt;
    const bool needF = nt == T_FULL && old != T_FULL;
    const bool needQ = nt == T_QUANT && old != T_QUANT && led == L_NONE;
    my_req[k] = (needF ? 1 : 0) | (needQ ? 2 : 0);
    my_nb[k] = G.bits_cfg == 42 ? (rq < half_q ? 4 : 2) : G.bits_cfg;
    if (old == T_FULL && nt != T_FULL) fown[my_fs[k]] = -2;   // vacated in this event
    if (nt == T_EVICTED && led != L_NONE) qown[my_qs[k]] = -1;
  }
  __syncthreads();

  // ---- free lists and request ranks: five flag prefix counts in one pass ----
  // The bf16 free list holds the slots free before this event first, then the
  // slots vacated in it, so promotions use a vacated slot (and must wait for
  // the quantization reading it) only once the spare slots are used up.
  int my_rankF[PER], my_rankQ[PER];
  int nfreeF, nfreeQ, nreqF, nreqQ;
  {
    bool fl[5][PER];
    int rk[5][PER], tots[5];
    const int km = max(kc, ko);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = tid + k * NT;
      const int fo = k < ko && i < G.n_fslots ? fown[i] : 0;
      fl[0][k] = fo == -1;
      fl[1][k] = k < ko && i < G.n_qslots && qown[i] < 0;
      fl[2][k] = (my_req[k] & 1) != 0;
      fl[3][k] = (my_req[k] & 2) != 0;
      fl[4][k] = fo == -2;
    }
    flag_scan<5>(fl, rk, tots, tmp, km);
    nfreeF = tots[0] + tots[4];
    nfreeQ = tots[1];
    nreqF = tots[2];
    nreqQ = tots[3];
    // free slot lists, ascending slot order within each group (sinfo / sb are free now)
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (k >= km) break;
      const int i = tid + k * NT;
      if (fl[0][k]) sinfo[rk[0][k]] = i;
      if (fl[4][k]) sinfo[tots[0] + rk[4][k]] = i;
      if (fl[1][k]) sb[rk[1][k]] = i;
      my_rankF[k] = rk[2][k];
      my_rankQ[k] = rk[3][k];
    }
  }
  int32_t* freeF = sinfo;
  int32_t* freeQ = sb;
  int32_t* sdep = sa;   // per bf16 slot: quantization entry reading it in this event, or -1
  for (int i = tid; i < G.n_fslots; i += NT) sdep[i] = -1;
  __syncthreads();

  // ---- apply: new slots, ledger states, work lists ----
  const int src_aged = a.prefill ? SRC_PROMPT : SRC_RING;
  int my_aux[PER], my_pl[PER];   // promotion / admission entry to write once slot dependencies are known
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = tid + k * NT;
    my_aux[k] = -1;
    my_pl[k] = -1;
    if (k >= kc || c >= n_cand) continue;
    const int w = my_w[k];
    const int old = my_old[k], nt = my_nt[k];
    int led = my_led[k];
    int fs = nt == T_FULL && old == T_FULL ? my_fs[k] : -1;
    int qs = my_qs[k];
    int nb = my_bits[k];
    if (my_req[k] & 1) {
      const int rk = my_rankF[k];
      if (rk < nfreeF) {
        fs = freeF[rk];
        fown[fs] = w;
        my_pl[k] = rk;
        if (old == T_QUANT) {
          led = L_DORMANT;
          atomicAdd(&sstat[ST_PROMO], 1);
        } else {
          atomicAdd(&sstat[ST_ADMIT], 1);
        }
      } else {
        set_error(counts, ERR_POOL);
      }
    }
    if (my_req[k] & 2) {
      const int rk = my_rankQ[k];
      if (rk < nfreeQ) {
        qs = freeQ[rk];
        qown[qs] = w;
        nb = my_nb[k];
        led = L_ACTIVE;
        int32_t* e = qlist + rk * kQEntry;
        e[0] = w;
        if (old == T_FULL) {
          e[1] = SRC_FSLOT;
          e[2] = my_fs[k];
          sdep[my_fs[k]] = rk;
        } else {
          e[1] = src_aged;
          e[2] = a.prefill ? w : w % G.NR;
        }
        e[3] = qs;
        e[4] = nb;
        e[5] = -1;
        atomicAdd(&sstat[ST_FIRSTQ], 1);
      } else {
        set_error(counts, ERR_POOL);
      }
    }
    if (nt == T_QUANT && old == T_FULL && led == L_DORMANT) {
      led = L_ACTIVE;
      atomicAdd(&sstat[ST_REACT], 1);
    }
    if (nt == T_EVICTED) {
      led = L_NONE;
      qs = -1;
      atomicAdd(&sstat[ST_EVICT], 1);
    }
    tier[w] = (int8_t)nt;
    ledger[w] = (int8_t)led;
    bits[w] = (int8_t)nb;
    fslot[w] = fs;
    qslot[w] = qs;
    my_fs[k] = fs;
    my_qs[k] = qs;
    my_bits[k] = nb;
    my_aux[k] = qs >= 0 ? (qs | (nb << 28)) : -1;
  }
  __syncthreads();
  // promotion / admission entries: one whose bf16 slot is being quantized away in
  // this event runs after that quantization (paired through the dep fields)
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (k >= kc) break;
    if (my_pl[k] < 0) continue;
    const int rk = my_pl[k], w = my_w[k], fs = my_fs[k];
    int32_t* e = plist + rk * kQEntry;
    e[0] = w;
    if (my_old[k] == T_QUANT) {
      e[1] = SRC_QSLOT; e[2] = my_qs[k]; e[4] = my_bits[k];
    } else {
      e[1] = src_aged; e[2] = a.prefill ? w : w % G.NR; e[4] = 0;
    }
    e[3] = fs;
    const int dep = sdep[fs];
    e[5] = dep;
    if (dep >= 0) qlist[dep * kQEntry + 5] = rk;
  }
  for (int i = tid; i < G.n_fslots; i += NT) fowner[i] = fown[i] < 0 ? -1 : fown[i];
  for (int i = tid; i < G.n_qslots; i += NT) qowner[i] = qown[i];

  // ---- rebuild the live list (window order) with its cost prefix ----
  // The split plans of the next decode steps are filled in on the way: the
  // attention splits the items (the live list, then plan_extra recent-region and
  // sink windows of cost cost_bf16) at the cuts ceil(u total / 4S), u = 0..4S, and
  // the wave of part u starts at the first item whose start cost reaches cut u.
  // The items' cost intervals (start, end] partition (0, total], so cut u >= 1 lies
  // in exactly one of them and part u starts at the item after it (cut 0: item 0).
  // Cut u lies in (start, end] <=> start 4S < u total <= end 4S.  One plan per
  // slot, each for its own number of windows after the list.
  int n_items, total_live;
  int32_t* s_pref = sinfo;   // LDS copy of the new list's refs (free once the work lists are written)
  const int S4 = 4 * G.n_split;
  // part u's first item in slot j: sown[j (S4 + 1) + u] (owner tables are written back)
  auto cover = [&](int j, int start, int end, int total, int next) {
    int32_t* s_first = sown + j * (S4 + 1);
    const int u_lo = (int)((uint32_t)start * (uint32_t)S4 / (uint32_t)total) + 1;
    const int u_hi = (int)((uint32_t)end * (uint32_t)S4 / (uint32_t)total);
    for (int u = u_lo; u <= u_hi; ++u) s_first[u] = next;
  };
  static_assert(kPlanSlots * (4 * 256 + 1) <= 2 * kMaxCand, "plan slots fit the owner tables");
  __syncthreads();
  {
    bool fl[3][PER];
    int rk[3][PER], tots[3];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int c = tid + k * NT;
      const bool in = k < kc && c < n_cand;
      fl[0][k] = in && my_nt[k] == T_FULL;
      fl[1][k] = in && my_nt[k] == T_QUANT && my_bits[k] == 4;
      fl[2][k] = in && my_nt[k] == T_QUANT && my_bits[k] != 4;
    }
    flag_scan<3>(fl, rk, tots, tmp, kc);
    n_items = tots[0] + tots[1] + tots[2];
    total_live = tots[0] * G.cost_bf16 + tots[1] * G.cost_q4 + tots[2] * G.cost_q2;
    int total[kPlanSlots];   // the planned steps' totals
#pragma unroll
    for (int j = 0; j < kPlanSlots; ++j) {
      total[j] = total_live + U.plan_extra[j] * G.cost_bf16;
      if (U.plan_t0[j] <= 0) continue;
      int32_t* s_first = sown + j * (S4 + 1);
      if (tid == 0) s_first[0] = 0;
      if (total[j] == 0)
        for (int u = tid; u <= S4; u += NT) s_first[u] = 0;
      for (int e = tid; e < U.plan_extra[j]; e += NT)   // recent-region and sink windows
        cover(j, total_live + e * G.cost_bf16, total_live + (e + 1) * G.cost_bf16, total[j], n_items + e + 1);
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (k >= kc) break;
      if (!(fl[0][k] || fl[1][k] || fl[2][k])) continue;
      const int pos = rk[0][k] + rk[1][k] + rk[2][k];
      const int kind = fl[0][k] ? KIND_BF16 : (fl[1][k] ? KIND_Q4 : KIND_Q2);
      const int slot = fl[0][k] ? my_fs[k] : my_qs[k];
      atomicAdd(&sstat[fl[0][k] ? ST_NF : (fl[1][k] ? ST_NQ4 : ST_NQ2)], 1);
      const int ref = (kind << 28) | slot;
      const int cost = rk[0][k] * G.cost_bf16 + rk[1][k] * G.cost_q4 + rk[2][k] * G.cost_q2;
      iwin[pos] = my_w[k];
      iref[pos] = ref;
      iaux[pos] = my_aux[k];
      iscore[pos] = my_sc[k];
      icost[pos] = cost;
      s_pref[pos] = ref;
#pragma unroll
      for (int j = 0; j < kPlanSlots; ++j)
        if (U.plan_t0[j] > 0) cover(j, cost, cost + item_cost(G, kind), total[j], pos + 1);
    }
    if (tid == 0) {
      icost[n_items] = total_live;
      counts[CNT_COST] = total_live;
    }
  }
  // list positions after the live windows hold the recent-region windows of the
  // next steps: their scores as they stand (windows not started yet: 0)
  for (int j = tid; n_items + j < G.max_items; j += NT) iscore[n_items + j] = j < G.NR ? ring_sc : 0.f;
  __syncthreads();
  if (tid == 0) {
    counts[CNT_ITEMS] = n_items;
    counts[CNT_QUANT] = nreqQ < nfreeQ ? nreqQ : nfreeQ;
    counts[CNT_PROMOTE] = nreqF < nfreeF ? nreqF : nfreeF;
  }
  if (tid < ST_N) stats[tid] = sstat[tid];

  // ---- split plan records: slot j, part u = 4 s + w ----
#pragma unroll
  for (int j = 0; j < kPlanSlots; ++j) {
    if (U.plan_t0[j] <= 0) continue;
    const int32_t* s_first = sown + j * (S4 + 1);
    int32_t* prec = (int32_t*)(ub + a.L.plan) + j * S4 * kPlanRec;
    for (int u = tid; u < S4; u += NT) {
      const int first = s_first[u];
      int32_t r[kPlanRefs];
#pragma unroll
      for (int k = 0; k < kPlanRefs; ++k) r[k] = first + k < n_items ? s_pref[first + k] : 0;
      static_assert(kPlanRec == 8, "two 16-byte stores per record");
      u32x4* q = (u32x4*)(prec + u * kPlanRec);
      q[0] = (u32x4){(uint32_t)first, (uint32_t)s_first[u + 1], (uint32_t)r[0], (uint32_t)r[1]};
      q[1] = (u32x4){(uint32_t)r[2], (uint32_t)r[3], (uint32_t)r[4], (uint32_t)r[5]};
    }
  }
  if (tid < 2 * kPlanSlots) {
    const int j = tid >> 1;
    counts[CNT_PLAN_T0 + tid] = (tid & 1) ? U.plan_t1[j] : U.plan_t0[j];
  }
}

// Manual single-window move (one thread): F -> Q (quantize once or reactivate)
// or Q -> F (promotion), with the same ledger rules as a routing event.
__global__ void k_manual_move(RetierArgs a, int seq, int window, int to_quant) {
  const Geometry& G = a.g;
  uint8_t* ub = a.unit[0].base + (int64_t)seq * a.L.unit_bytes;
  int8_t* tier = (int8_t*)(ub + a.L.tier);
  int8_t* ledger = (int8_t*)(ub + a.L.ledger);
  int8_t* bits = (int8_t*)(ub + a.L.bits);
  int32_t* fslot = (int32_t*)(ub + a.L.fslot);
  int32_t* qslot = (int32_t*)(ub + a.L.qslot);
  int32_t* fowner = (int32_t*)(ub + a.L.fowner);
  int32_t* qowner = (int32_t*)(ub + a.L.qowner);
  int32_t* iwin = (int32_t*)(ub + a.L.item_win);
  int32_t* iref = (int32_t*)(ub + a.L.item_ref);
  int32_t* icost = (int32_t*)(ub + a.L.item_cost);
  int32_t* iaux = (int32_t*)(ub + a.L.item_aux);
  int32_t* qlist = (int32_t*)(ub + a.L.qlist);
  int32_t* plist = (int32_t*)(ub + a.L.plist);
  int32_t* counts = (int32_t*)(ub + a.L.counts);
  const int w = window;
  counts[CNT_QUANT] = 0;
  counts[CNT_PROMOTE] = 0;
  int kind = -1, slot = -1;
  if (to_quant) {
    const int fs = fslot[w];
    if (ledger[w] == L_DORMANT) {
      ledger[w] = L_ACTIVE;
    } else {
      int qs = -1;
      for (int i = 0; i < G.n_qslots && qs < 0; ++i)
        if (qowner[i] < 0) qs = i;
      if (qs < 0) { set_error(counts, ERR_POOL); return; }
      const int nb = G.bits_cfg == 42 ? 4 : G.bits_cfg;
      qowner[qs] = w;
      qslot[w] = qs;
      bits[w] = (int8_t)nb;
      ledger[w] = L_ACTIVE;
      int32_t* e = qlist;
      e[0] = w; e[1] = SRC_FSLOT; e[2] = fs; e[3] = qs; e[4] = nb; e[5] = -1;
      counts[CNT_QUANT] = 1;
    }
    fowner[fs] = -1;
    fslot[w] = -1;
    tier[w] = T_QUANT;
    kind = bits[w] == 4 ? KIND_Q4 : KIND_Q2;
    slot = qslot[w];
  } else {
    int fs = -1;
    for (int i = 0; i < G.n_fslots && fs < 0; ++i)
      if (fowner[i] < 0) fs = i;
    if (fs < 0) { set_error(counts, ERR_POOL); return; }
    fowner[fs] = w;
    fslot[w] = fs;
    ledger[w] = L_DORMANT;
    tier[w] = T_FULL;
    int32_t* e = plist;
    e[0] = w; e[1] = SRC_QSLOT; e[2] = qslot[w]; e[3] = fs; e[4] = bits[w]; e[5] = -1;
    counts[CNT_PROMOTE] = 1;
    kind = KIND_BF16;
    slot = fs;
  }
  // the window keeps its position in the live list; refresh its entry and the cost prefix
  const int n = counts[CNT_ITEMS];
  int run = 0;
  const int aux = qslot[w] >= 0 ? (qslot[w] | (bits[w] << 28)) : -1;
  for (int i = 0; i < n; ++i) {
    if (iwin[i] == w) {
      iref[i] = (kind << 28) | slot;
      iaux[i] = aux;
    }
    icost[i] = run;
    run += item_cost(G, iref[i] >> 28);
  }
  icost[n] = run;
  counts[CNT_COST] = run;
  for (int j = 0; j < kPlanSlots; ++j) {   // the split plans no longer match the list
    counts[CNT_PLAN_T0 + 2 * j] = -1;
    counts[CNT_PLAN_T1 + 2 * j] = -2;
  }
}

// Key-norm scores of the prompt windows (appendix, key-norm equation):
// S(w) = -(1/W) sum over the window's prompt tokens of |k_t|, |k_t| the L2 norm
// of token t's key over all KV heads.  One workgroup per (window, sequence);
// thread (token, head) sums its 128 squares, heads then tokens are summed in a
// fixed order.
__global__ __launch_bounds__(256) void k_key_norm_init(KeyNormArgs a) {
  const Geometry& G = a.g;
  const int w = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  __shared__ float ssq[256];
  __shared__ float snorm[64];
  const int t0 = G.sink + w * G.W, t1 = min(t0 + G.W, a.T);
  const int nt = t1 - t0;
  for (int base = 0; base < G.W; base += 256 / G.H_kv) {
    const int lt = base + tid / G.H_kv, g = tid % G.H_kv;
    float sq = 0.f;
    if (tid < (256 / G.H_kv) * G.H_kv && lt < nt) {
      const u32x4* row = (const u32x4*)(a.k + (((int64_t)b * G.H_kv + g) * a.T + t0 + lt) * kHeadDim);
#pragma unroll 4
      for (int i = 0; i < kHeadDim / 8; ++i) {
        const u32x4 x = row[i];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float lo = __uint_as_float(x[j] << 16), hi = __uint_as_float(x[j] & 0xFFFF0000u);
          sq = fmaf(lo, lo, sq);
          sq = fmaf(hi, hi, sq);
        }
      }
    }
    ssq[tid] = sq;
    __syncthreads();
    if (tid < 256 / G.H_kv && base + tid < G.W) {
      float s2 = 0.f;
      for (int h = 0; h < G.H_kv; ++h) s2 += ssq[tid * G.H_kv + h];
      snorm[base + tid] = base + tid < nt ? sqrtf(s2) : 0.f;
    }
    __syncthreads();
  }
  if (tid == 0) {
    float s = 0.f;
    for (int t = 0; t < G.W; ++t) s += snorm[t];
    a.out[(int64_t)b * a.n_init + w] = -s / (float)G.W;
  }
}

// p-norm ranking: the prompt's initial scores are the first routing period's
// attention u_0, entering the score as u_0^p (appendix, p-norm equation).  A
// negative score yields NaN, which the re-rank kernel reports as non-finite.
__global__ __launch_bounds__(256) void k_score_pow(ScorePowArgs a) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= a.n) return;
  const float x = a.in[i];
  a.out[i] = x >= 0.f ? powf(x, a.p) : __builtin_nanf("");
}

// Ordering of the routing stream after the cache stream without a queue-level
// wait (a barrier packet waiting on another queue's signal measurably delays the
// cache stream's own dispatches here).  The cache stream publishes a sequence
// number after the work a routing batch must follow; kernel completion makes that
// work visible device-wide, and the release store orders the number after it.
// The routing stream starts each batch with a one-wave wait for the number
// (acquire); past `ticks` of the wall clock (or a poll cap, should the clock not
// advance) it raises the gate failure word instead, and the batch's re-rank and
// migration kernels then do nothing.
__global__ void k_gate_publish(uint64_t* seq, uint64_t value, int32_t* clear) {
  if (threadIdx.x != 0) return;
  if (clear) __hip_atomic_store(clear, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(seq, value, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void k_gate_wait(const uint64_t* seq, uint64_t value, int32_t* fail, int64_t ticks) {
  if (threadIdx.x != 0) return;
  const int64_t t0 = (int64_t)wall_clock64();
  for (int64_t polls = 0; __hip_atomic_load(seq, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < value;
       ++polls) {
    if ((int64_t)wall_clock64() - t0 > ticks || polls > kGateMaxPolls) {
      __hip_atomic_store(fail, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    __builtin_amdgcn_s_sleep(16);
  }
}

hipError_t launch_gate_publish(uint64_t* seq, uint64_t value, int32_t* clear, hipStream_t st) {
  hipLaunchKernelGGL(k_gate_publish, dim3(1), dim3(64), 0, st, seq, value, clear);
  return hipGetLastError();
}
hipError_t launch_gate_wait(const uint64_t* seq, uint64_t value, int32_t* fail, int64_t ticks,
                            hipStream_t st) {
  hipLaunchKernelGGL(k_gate_wait, dim3(1), dim3(64), 0, st, seq, value, fail, ticks);
  return hipGetLastError();
}

// State initialisation of every unit block (grid-stride over units).
__global__ void k_init_units(Geometry G, UnitLayout L, uint8_t* base, int n_units) {
  for (int u = blockIdx.x; u < n_units; u += gridDim.x) {
    uint8_t* ub = base + (int64_t)u * L.unit_bytes;
    for (int w = threadIdx.x; w < G.nwc; w += blockDim.x) {
      ((int8_t*)(ub + L.tier))[w] = T_UNUSED;
      ((int8_t*)(ub + L.ledger))[w] = L_NONE;
      ((int8_t*)(ub + L.bits))[w] = 0;
      ((int32_t*)(ub + L.fslot))[w] = -1;
      ((int32_t*)(ub + L.qslot))[w] = -1;
      ((float*)(ub + L.score))[w] = 0.f;
      if (G.score_mode == kScorePnorm) ((float2*)(ub + L.pnorm))[w] = make_float2(0.f, 0.f);
    }
    for (int i = threadIdx.x; i < G.n_fslots; i += blockDim.x) ((int32_t*)(ub + L.fowner))[i] = -1;
    for (int i = threadIdx.x; i < G.n_qslots; i += blockDim.x) ((int32_t*)(ub + L.qowner))[i] = -1;
    for (int i = threadIdx.x; i < CNT_N; i += blockDim.x) ((int32_t*)(ub + L.counts))[i] = 0;
    for (int i = threadIdx.x; i < ST_N; i += blockDim.x) ((int32_t*)(ub + L.stats))[i] = 0;
    if (threadIdx.x == 0) ((int32_t*)(ub + L.item_cost))[0] = 0;
    // recent-ring and sink slots start as zeros (partial windows read them)
    const int64_t nz = (int64_t)(G.NR + G.NS) * G.fslot_bytes / 16;
    u32x4* z = (u32x4*)(ub + L.ring);
    for (int64_t i = threadIdx.x; i < nz; i += blockDim.x) z[i] = (u32x4){0, 0, 0, 0};
  }
}

hipError_t launch_key_norm_init(const KeyNormArgs& a, hipStream_t st) {
  if (a.n_init <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_key_norm_init, dim3(a.n_init, a.g.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_score_pow(const ScorePowArgs& a, hipStream_t st) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_score_pow, dim3((a.n + 255) / 256), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_retier(const RetierArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_retier, dim3(a.g.B, a.n_units), dim3(kRetierThreads), 0, st, a);
  return hipGetLastError();
}
hipError_t launch_manual_move(const RetierArgs& a, int seq, int window, int to_quant, hipStream_t st) {
  hipLaunchKernelGGL(k_manual_move, dim3(1), dim3(1), 0, st, a, seq, window, to_quant);
  return hipGetLastError();
}
hipError_t launch_init_units(const Geometry& g, const UnitLayout& L, uint8_t* base, int n_units,
                             hipStream_t st) {
  hipLaunchKernelGGL(k_init_units, dim3(n_units < 1024 ? n_units : 1024), dim3(256), 0, st, g, L,
                     base, n_units);
  return hipGetLastError();
}

}  // namespace qv
