// Tier-aware split-K decode attention and the split merge / window-score pass.
//
// Decode attention of each query head over the accessible tokens (QEvict
// Sec. 4.1): sink and recent tokens and Full windows in bf16, Quantized
// windows as z + s c with the codes expanded in registers.  The pass also
// yields, per (query head, window), the window's softmax mass relative to a
// reference maximum, which the merge turns into the exact attention mass the
// window received and adds, averaged over the query heads, to the window's
// cumulative score (Sec. 4.2, cumulative window score equation).
//
// Work decomposition: one workgroup per (sequence, KV head, split); the live
// windows of a sequence form a list in window order, cut into splits of equal
// estimated cost; the 4 waves of a workgroup take the split's windows round
// robin.  A wave handles the G = H_q / H_kv query heads of its KV head at once:
//   S^T[token][head] = K . Q^T   (16x16x32 MFMA, tokens as rows, heads padded to 16)
//   O[head][chan]   += P . V     (16x16x32 MFMA; P taken straight from S^T's lanes)
// Quantized keys use S^T = codes . (q*s)^T + q.z with q*s split into two fp16
// halves (hi + lo represent the product exactly), so the logits keep fp32
// accuracy; quantized values are expanded to fp16 z + s c before P . V.
#include "qv_device.h"

namespace qv {

__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_f16(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
// 16x16x16 MFMAs of the P.V product of 8-token windows (k = 16 tokens of which
// the window fills 8): A lane 16 q + r holds A[r][4 q + j], B lane holds B[4 q + j][r]
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4 mfma16_bf16(bf16x4 a, bf16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16_f16(f16x4 a, f16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ u32x4 ld16(const void* p) { return *(const u32x4*)p; }
// Completes this wave's LDS operations before the next ones (LDS traffic of one
// wave is ordered; the memory clobber keeps the compiler from moving accesses).
__device__ __forceinline__ void wave_sync_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// sum over the 16 lanes of a row with DPP (quad swaps, half-row and row mirrors)
__device__ __forceinline__ float row16_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false));
  return x;
}

// 8 codes of one (entry, lane) as exact fp16 integers; ee = entry slot in its word
template <int BITS>
__device__ __forceinline__ f16x8 unpack_codes(uint32_t w, int ee) {
  constexpr uint32_t mask = BITS == 4 ? 0x000F000Fu : 0x00030003u;
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t x = ((w >> (BITS * (4 * ee + i))) & mask) | 0x64006400u;   // 1024 + code
    f16x2 h = __builtin_bit_cast(f16x2, x) - (f16x2){(_Float16)1024.0f, (_Float16)1024.0f};
    r[2 * i] = h[0];
    r[2 * i + 1] = h[1];
  }
  return r;
}

template <int BITS>
__device__ __forceinline__ uint32_t code_word(const uint32_t* words, int e, int* ee) {
  constexpr int per = 4 / BITS;
  *ee = e % per;
  return words[e / per];
}

struct WaveState {
  float m, l;      // running max (log2 domain) and sum for head r of this lane
  f32x4 o[8];      // O rows 4*qg + v, channels 16*cb + r
};

// Online-softmax update for one window; returns the probabilities in p[tb][v]
// relative to the wave's running reference maximum and records the window's
// (reference, sum) pair.  The reference is raised (and O rescaled) only when a
// window's maximum exceeds it by more than 2^8, so probabilities stay <= 2^8
// and most windows skip the rescale.
constexpr float kRescaleSlack = 8.0f;

template <int TB, int NHS>
__device__ __forceinline__ void softmax_window(const f32x4 (&acc)[TB], float bias, int ntok,
                                               float scale_log2, int qg, WaveState& st,
                                               float (&p)[TB][4], float* m_out, float* l_out) {
  float x[TB][4];
  float mw = -INFINITY;
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int t = 16 * tb + 4 * qg + v;
      float y = (acc[tb][v] + bias) * scale_log2;
      y = t < ntok ? y : -INFINITY;
      x[tb][v] = y;
      mw = fmaxf(mw, y);
    }
  mw = rows_max(mw);
  if (__builtin_amdgcn_ballot_w64(mw > st.m + kRescaleSlack) != 0) {
    const float m_new = fmaxf(st.m, mw);
    const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
    st.l *= alpha;
    st.m = m_new;
    // O rows 4*qg + v belong to head 4*qg + v, whose alpha lane r = 4*qg + v holds
    if constexpr (NHS == 1) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float av = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alpha), v));
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) st.o[cb][v] *= av;
      }
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float av = __shfl(alpha, 4 * qg + v);
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) st.o[cb][v] *= av;
      }
    }
  }
  float lw = 0.f;
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      p[tb][v] = __builtin_amdgcn_exp2f(x[tb][v] - st.m);
      lw += p[tb][v];
    }
  lw = rows_sum(lw);
  st.l += lw;
  *m_out = st.m;
  *l_out = lw;
}

// Per-window operands in registers, split into the part the QK^T phase reads
// (K) and the part the P.V phase reads (V).
//   bf16 window: K chunks (tb, kb) at kh.d[tb * 4 + kb]; V chunks (kt, cb) at vh.d[kt * 8 + cb]
//   quantized:   K codes kh.d[0 .. NC), K scale / zero (compact) kh.d[NC], kh.d[NC + 1];
//                V codes vh.d[0 .. NC), V scale / zero per (kt, vg) at vh.d[NC + 2 (kt NG + vg)] (+1)
//   8-token window: bf16 K chunks kb at kh.d[kb] (lanes r < 8), V chunks cp at
//                vh.d[cp] (lanes q < 2); quantized K codes kh.d[0], compact key
//                scale / zero kh.d[1], kh.d[2]; V codes vh.d[0], V scale / zero of
//                value group g for the lane's 4 tokens vh.d[1 + g]
// (entries of code registers before the compact key meta, and its index)
template <int W>
constexpr int key_code_regs() { return W == 8 ? 1 : W / 16; }
// 16-token row tiles of a window's QK^T (an 8-token window fills half of one)
template <int W>
constexpr int row_tiles() { return W == 8 ? 1 : W / 16; }
template <int W, bool ROPE = false>
struct KHalf {
  static constexpr int N = W == 8 ? 4 : W / 4;
  u32x4 d[N];
};
template <int W>
struct VHalf {
  static constexpr int N = W == 8 ? 5 : (W == 32 ? 10 : 16);
  u32x4 d[N];
};

struct ItemInfo {
  const uint8_t* p;
  int kind, ntok, it;
  int win;   // window index of a live-list item (RoPE positions), else -1
  bool open;
};

// RQ: the key scale / zero registers hold channels 32 (r >> 2) + 8 qg .. + 7 (the
// block the lane forms q*s for in registers) instead of 8 r .. 8 r + 7
template <int W, bool ROPE, bool RQ = false>
__device__ __forceinline__ void fetch_k(const ItemInfo& in, KHalf<W, ROPE>& kh, int lane, int r,
                                        const Geometry& G) {
  constexpr int TB = W / 16, NC = W / 16;
  const uint8_t* p = in.p;
  if constexpr (W == 8) {
    const bool row = r < 8;   // lanes of the window's 8 token rows
    const int qg = lane >> 4;
    if (in.kind == KIND_BF16) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) kh.d[kb] = row ? ld16(p + ((kb * 4 + qg) * 8 + r) * 16) : (u32x4){0, 0, 0, 0};
    } else {
      kh.d[3] = (u32x4){0, 0, 0, 0};
      if (in.kind == KIND_Q4) {
        kh.d[0] = row ? ld16(p + (qg * 8 + r) * 16) : (u32x4){0, 0, 0, 0};
      } else {
        const uint2 c2 = row ? *(const uint2*)(p + (qg * 8 + r) * 8) : make_uint2(0, 0);
        kh.d[0] = (u32x4){c2.x, c2.y, 0, 0};
      }
      const uint8_t* mk = p + meta_k_off(G);
      kh.d[1] = ld16(mk + 16 * r);
      kh.d[2] = ld16(mk + 256 + 16 * r);
    }
    return;
  } else if (in.kind == KIND_BF16) {
#pragma unroll
    for (int i = 0; i < 4 * TB; ++i) kh.d[i] = ld16(p + (i * 64 + lane) * 16);
  } else {
    const int nld = in.kind == KIND_Q4 ? NC : NC / 2;
    // every register of the buffer is defined on both paths (keeps it out of scratch)
#pragma unroll
    for (int i = 0; i < KHalf<W, ROPE>::N; ++i) kh.d[i] = (u32x4){0, 0, 0, 0};
#pragma unroll
    for (int m = 0; m < NC; ++m)
      if (m < nld) kh.d[m] = ld16(p + (m * 64 + lane) * 16);
    const uint8_t* mk = p + meta_k_off(G);
    const int mo = RQ ? 64 * (r >> 2) + 16 * (lane >> 4) : 16 * r;
    kh.d[NC] = ld16(mk + mo);
    kh.d[NC + 1] = ld16(mk + 256 + mo);
    if constexpr (ROPE) {   // (cos, sin) of the window's first position, pairs 8 (r & 7) .. + 7
      static_assert(KHalf<W, ROPE>::N >= W / 16 + 6, "spare registers for the rotation");
      const float* c0 = G.rope + 2 * ((int64_t)(G.sink + in.win * W) * (kHeadDim / 2) + 8 * (r & 7));
#pragma unroll
      for (int k = 0; k < 4; ++k) kh.d[NC + 2 + k] = ld16(c0 + 4 * k);
    }
  }
}

template <int W>
__device__ __forceinline__ void fetch_v(const ItemInfo& in, VHalf<W>& vh, int lane, int qg,
                                        const Geometry& G) {
  constexpr int KT = W / 32, NC = W / 16, NG = kHeadDim / W;
  const uint8_t* p = in.p;
  if constexpr (W == 8) {
    const bool col = qg < 2;   // lanes of the window's 8 tokens in the B operand
    const int r = lane & 15;
    if (in.kind == KIND_BF16) {
      const int64_t vbase = (int64_t)W * kHeadDim * 2;
#pragma unroll
      for (int cp = 0; cp < 4; ++cp)
        vh.d[cp] = col ? ld16(p + vbase + ((cp * 2 + qg) * 16 + r) * 16) : (u32x4){0, 0, 0, 0};
      vh.d[4] = (u32x4){0, 0, 0, 0};
    } else {
      if (in.kind == KIND_Q4) {
        vh.d[0] = col ? ld16(p + G.qcodes_bytes + (qg * 16 + r) * 16) : (u32x4){0, 0, 0, 0};
      } else {
        const uint2 c2 = col ? *(const uint2*)(p + G.qcodes_bytes + (qg * 16 + r) * 8) : make_uint2(0, 0);
        vh.d[0] = (u32x4){c2.x, c2.y, 0, 0};
      }
#pragma unroll
      for (int vg = 0; vg < 4; ++vg)
        vh.d[1 + vg] = col ? ld16(p + meta_v_off(G) + ((qg * 4 + vg) * 16)) : (u32x4){0, 0, 0, 0};
    }
    return;
  } else if (in.kind == KIND_BF16) {
    const int64_t vbase = (int64_t)W * kHeadDim * 2;
#pragma unroll
    for (int i = 0; i < VHalf<W>::N; ++i)
      vh.d[i] = i < 8 * KT ? ld16(p + vbase + (i * 64 + lane) * 16) : (u32x4){0, 0, 0, 0};
  } else {
    const int nld = in.kind == KIND_Q4 ? NC : NC / 2;
#pragma unroll
    for (int i = 0; i < VHalf<W>::N; ++i) vh.d[i] = (u32x4){0, 0, 0, 0};
#pragma unroll
    for (int m = 0; m < NC; ++m)
      if (m < nld) vh.d[m] = ld16(p + G.qcodes_bytes + (m * 64 + lane) * 16);
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int vg = 0; vg < NG; ++vg) {
        const uint8_t* pm = p + meta_v_off(G) + ((kt * 4 + qg) * NG + vg) * 32;
        vh.d[NC + (kt * NG + vg) * 2] = ld16(pm);
        vh.d[NC + 1 + (kt * NG + vg) * 2] = ld16(pm + 16);
      }
  }
}

// ---- 8-token windows: two windows per pass of the latency chain ----
//
// With at most four query heads per KV head the 16 columns of the QK^T tile
// have room for the heads of two windows: window A's heads in columns 0..3 and
// window B's in columns 4..7, A's keys in rows 0..7 and B's in rows 8..15.  A
// column keeps the logits of its own window's rows (the others are masked), so
// each column block is an online softmax of its own (a stream), and P.V
// (K = 16 tokens: A's in lane groups 0, 1, B's in 2, 3) accumulates stream 0
// into O rows 0..3 and stream 1 into rows 4..7; the two streams of a head are
// merged at the end of the run.  A pass -- slot wait, operand reads, MFMAs,
// row max, exponentials, sums -- so serves two windows.  Consecutive windows of
// a run are paired when they are of one kind.
//
// Both records of the next pair go straight from their pools into the wave's
// LDS slot (direct global-to-LDS loads, 16 bytes a lane; the instruction writes
// lane L's bytes at slot row + 16 L) while the current pair is computed, without
// registers to hold them; the records are copied as they lie in their pools --
// 4 KiB for a bf16 window, at most 2 KiB for a quantized record.  No
// register-destination load is pending while slot loads are in flight (the
// compiler would then wait for all of them).  With 32-token windows a wave has
// about two windows, and issuing the next window's loads and copying it out of
// the LDS cost as much as the overlap gains, so those keep their windows in
// registers only.
template <int W, int NHS, bool ROPE>
constexpr bool use_slot() { return NHS == 1 && !ROPE && W == 8; }
// q*s of a quantized window formed in registers (64-token windows, at most four
// query heads per KV head): lane (q, r) forms channel block r >> 2 of column r & 3,
// and lane r takes the other blocks of its column from lanes r + 4, r + 8 and
// r + 12 with row rotations (columns 4..15 repeat heads 0..3; their logits are
// computed and never used).  With 32-token windows the LDS staging measured
// slightly faster, so those keep it.
template <int W, int NHS, bool ROPE>
constexpr bool use_reg_qs() { return NHS == 1 && !ROPE && W == 64; }

// lane r of each 16-lane row takes lane (r + 16 - N) mod 16 (row rotation right by N)
template <int N>
__device__ __forceinline__ u32x4 row_ror(u32x4 v) {
  u32x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v[i], 0x120 + N, 0xF, 0xF, false);
  return o;
}
constexpr int kPairSlot = 4 * 1024;   // LDS bytes per window of a pair

__device__ __forceinline__ void dma16(const void* g, uint8_t* lds_row) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds_row, 16, 0, 0);
}

// bytes of the item's record: a bf16 window (keys then values), or a quantized
// record (key codes, value codes, key scale / zero, value scale / zero)
template <int W>
__device__ __forceinline__ int slot_record_bytes(const ItemInfo& in, const Geometry& G) {
  return in.kind == KIND_BF16 ? 2 * W * kHeadDim * 2 : (int)G.qrec_bytes;
}

__device__ __forceinline__ void issue_record(const ItemInfo& in, uint8_t* dst, int lane, const Geometry& G) {
  const int n = slot_record_bytes<8>(in, G);
#pragma unroll
  for (int row = 0; row < kPairSlot / 1024; ++row) {
    if (row * 1024 >= n) break;   // uniform
    if (row * 1024 + lane * 16 < n) dma16(in.p + row * 1024 + lane * 16, dst + row * 1024);
  }
}

// Operand registers of a pair, gathered from the slot: K rows r (window r >> 3,
// token r & 7), V lane groups qg (window qg >> 1, tokens 4 (qg & 1) ..); lanes of
// an absent window B read zeros.  Quantized windows: the B operand q*s of the
// lane's column (head r & 3 of window (r >> 2) & 1, channels 32 kb + 8 qg + i)
// split into exact fp16 hi + lo, and the column's bias q.z.
__device__ __forceinline__ void read_pair(int kind, bool pb, const uint8_t* slot, KHalf<8, false>& kh,
                                          VHalf<8>& vh, f16x8 (&qhi)[4], f16x8 (&qlo)[4], float* bias,
                                          const bf16x8 (&qop)[4], int r, int qg, const Geometry& G) {
  // Every read is unconditional (all addresses lie in the slot; lanes of an
  // absent window read stale bytes and select zeros), so the reads issue back
  // to back and one wait covers them.
  const u32x4 z = {0, 0, 0, 0};
  auto rd = [&](const uint8_t* s, int off) { return *(const u32x4*)(s + off); };
  auto sel = [&](bool c, u32x4 v) {
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = c ? v[i] : 0u;
    return o;
  };
  const bool krow = r < 8 || pb, vcol = qg < 2 || pb;
  const uint8_t* ks = slot + (r >= 8 ? kPairSlot : 0);
  const uint8_t* vs = slot + (qg >= 2 ? kPairSlot : 0);
  const int rr = r & 7, qq = qg & 1;
  if (kind == KIND_BF16) {
    const int vbase = 8 * kHeadDim * 2;
    u32x4 kv[4], vv[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) kv[kb] = rd(ks, ((kb * 4 + qg) * 8 + rr) * 16);
#pragma unroll
    for (int cp = 0; cp < 4; ++cp) vv[cp] = rd(vs, vbase + ((cp * 2 + qq) * 16 + r) * 16);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) kh.d[kb] = sel(krow, kv[kb]);
#pragma unroll
    for (int cp = 0; cp < 4; ++cp) vh.d[cp] = sel(vcol, vv[cp]);
    vh.d[4] = z;
    *bias = 0.f;
    return;
  }
  // codes: 16 bytes a lane (int4), 8 (int2: the upper half of the read is the
  // next lane's and is dropped)
  const bool q4 = kind == KIND_Q4;
  const int qc = (int)G.qcodes_bytes, mk = (int)meta_k_off(G), mv = (int)meta_v_off(G);
  const int cb = q4 ? 16 : 8;
  const u32x4 kc = rd(ks, (qg * 8 + rr) * cb);
  const u32x4 vc = rd(vs, qc + (qq * 16 + r) * cb);
  u32x4 vm[4];
#pragma unroll
  for (int vg = 0; vg < 4; ++vg) vm[vg] = rd(vs, mv + (qq * 4 + vg) * 16);
  // q*s of column c = r & 7 (head c & 3 of window c >> 2): lanes r < 8 form
  // channel blocks kb = 0, 1 and lanes r + 8 blocks 2, 3 of the same column, whose
  // halves lane r then takes with a half-row rotation (lanes r >= 8 keep operands
  // of masked columns)
  const int jc = (r >> 2) & 1, kb0 = (r >> 3) * 2;
  const bool cval = jc == 0 || pb;
  const uint8_t* cs = slot + (jc ? kPairSlot : 0);
  u32x4 s4[2], z4[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    s4[k] = rd(cs, mk + 64 * (kb0 + k) + 16 * qg);         // key scales
    z4[k] = rd(cs, mk + 256 + 64 * (kb0 + k) + 16 * qg);   // key zero points
  }
  const uint32_t hm = q4 ? ~0u : 0u;
  kh.d[0] = sel(krow, (u32x4){kc[0], kc[1], kc[2] & hm, kc[3] & hm});
  vh.d[0] = sel(vcol, (u32x4){vc[0], vc[1], vc[2] & hm, vc[3] & hm});
#pragma unroll
  for (int vg = 0; vg < 4; ++vg) vh.d[1 + vg] = sel(vcol, vm[vg]);
  float bsum = 0.f;
  u32x4 mh[2], ml[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const u32x4 sk = sel(cval, s4[k]), zk = sel(cval, z4[k]);
    const u32x4 qb = __builtin_bit_cast(u32x4, r < 8 ? qop[k] : qop[2 + k]);
    f16x8 hi8, lo8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float qv = __uint_as_float((i & 1) ? (qb[i >> 1] & 0xFFFF0000u) : (qb[i >> 1] << 16));
      const float sv = (float)__builtin_bit_cast(_Float16, (uint16_t)(sk[i >> 1] >> (16 * (i & 1))));
      const float zv = (float)__builtin_bit_cast(_Float16, (uint16_t)(zk[i >> 1] >> (16 * (i & 1))));
      const float qs = qv * sv;   // exact: 8-bit x 11-bit significands
      const _Float16 h = (_Float16)qs;
      hi8[i] = h;
      lo8[i] = (_Float16)(qs - (float)h);
      bsum = fmaf(qv, zv, bsum);
    }
    mh[k] = __builtin_bit_cast(u32x4, hi8);
    ml[k] = __builtin_bit_cast(u32x4, lo8);
  }
  auto ror8 = [](u32x4 v) {   // lane r takes lane r ^ 8 of its 16-lane row
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v[i], 0x128, 0xF, 0xF, false);
    return o;
  };
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    qhi[k] = __builtin_bit_cast(f16x8, mh[k]);
    qlo[k] = __builtin_bit_cast(f16x8, ml[k]);
    qhi[2 + k] = __builtin_bit_cast(f16x8, ror8(mh[k]));
    qlo[2 + k] = __builtin_bit_cast(f16x8, ror8(ml[k]));
  }
  bsum += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(bsum), 0x128, 0xF, 0xF, false));
  *bias = rows_sum(bsum);   // q . z of the column over its 128 channels
}

// The open window takes this step's key and value (and stores them into its
// ring slot); it is the pair's window j.
__device__ __forceinline__ void patch_open8(const ItemInfo& in, int j, KHalf<8, false>& kh, VHalf<8>& vh,
                                            const AttnArgs& a, int b, int g, int qg, int r) {
  const Geometry& G = a.g;
  const int pos = in.ntok - 1;
  uint8_t* pw = const_cast<uint8_t*>(in.p);
  const uint16_t* kn = a.k_new + ((int64_t)b * G.H_kv + g) * kHeadDim;
  const bool krow = r == 8 * j + pos;   // lanes of the token's key row
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const u32x4 v = ld16(kn + 32 * kb + 8 * qg);
#pragma unroll
    for (int i = 0; i < 4; ++i) kh.d[kb][i] = krow ? v[i] : kh.d[kb][i];
    if (krow) *(u32x4*)(pw + ((kb * 4 + qg) * 8 + pos) * 16) = v;
  }
  // value: element jp of the lanes of group 2 j + qp
  const uint16_t* vn = a.v_new + ((int64_t)b * G.H_kv + g) * kHeadDim;
  const int qp = pos >> 2, jp = pos & 3;
  const bool vgrp = qg == 2 * j + qp;
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) {
    const uint32_t val = vn[16 * cb + r];
    if (vgrp) *(uint16_t*)(pw + v_elem_off(8, pos, 16 * cb + r)) = (uint16_t)val;
    const int wi = (cb & 1) * 2 + (jp >> 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t wv = vh.d[cb >> 1][i];
      const uint32_t lo = (wv & 0xFFFF0000u) | val, hi = (wv & 0x0000FFFFu) | (val << 16);
      vh.d[cb >> 1][i] = (vgrp && i == wi) ? ((jp & 1) ? hi : lo) : wv;
    }
  }
}

// QK^T and the online-softmax update of a pair: the lane's probabilities of
// column r (rows 4 qg .. + 3) in p, the column's sum in *lw.  Masked entries
// are -inf, and a stream without any row yet keeps reference -inf and sum 0.
__device__ __forceinline__ void pair_k(int kind, bool pb, int ntA, int ntB, const KHalf<8, false>& kh,
                                       const bf16x8 (&qop)[4], const f16x8 (&qhi)[4],
                                       const f16x8 (&qlo)[4], float bias, float scale_log2, int qg,
                                       int r, WaveState& st, float (&p)[4], float* lw_out) {
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (kind == KIND_BF16) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) acc = mfma_bf16(__builtin_bit_cast(bf16x8, kh.d[kb]), qop[kb], acc);
  } else {
    const bool q4 = kind == KIND_Q4;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const f16x8 cv = q4 ? unpack_codes<4>(kh.d[0][kb], 0) : unpack_codes<2>(kh.d[0][kb >> 1], kb & 1);
      acc = mfma_f16(cv, qhi[kb], acc);
      acc = mfma_f16(cv, qlo[kb], acc);
    }
  }
  const int jc = (r >> 2) & 1;
  const bool cval = r < 8 && (jc == 0 || pb) && (qg >> 1) == jc;   // rows of the column's window
  const int ntok = jc ? ntB : ntA;
  float x[4];
  float mw = -INFINITY;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const bool ok = cval && 4 * (qg & 1) + v < ntok;
    x[v] = ok ? (acc[v] + bias) * scale_log2 : -INFINITY;
    mw = fmaxf(mw, x[v]);
  }
  mw = rows_max(mw);
  if (__builtin_amdgcn_ballot_w64(mw > st.m + kRescaleSlack) != 0) {
    const float m_new = fmaxf(st.m, mw);
    const float alpha = m_new == st.m ? 1.f : __builtin_amdgcn_exp2f(st.m - m_new);
    st.l *= alpha;
    st.m = m_new;
    // O row 4 qg + v: the alpha of lane 4 qg + v (rows 8..15 stay zero)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float a0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alpha), v));
      const float a1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alpha), 4 + v));
      const float av = qg == 0 ? a0 : a1;
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) st.o[cb][v] *= av;
    }
  }
  float lw = 0.f;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    p[v] = x[v] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(x[v] - st.m);
    lw += p[v];
  }
  lw = rows_sum(lw);
  st.l += lw;
  *lw_out = lw;
}

// P.V of a pair (16x16x16 MFMAs: the A operand is the lane's four
// probabilities of column r, the B operand the values of tokens 4 qg .. + 3),
// then the windows' statistics: (m_w, l_w) of stream j, head h from lane 4 j + h.
__device__ __forceinline__ void pair_v(int kind, bool pb, int itA, int itB, int ntA, int ntB, VHalf<8>& vh,
                                       WaveState& st, const float (&p)[4], float lw, const AttnArgs& a,
                                       int g, int qg, int r, float2* mref) {
  const Geometry& G = a.g;
  if (kind == KIND_BF16) {
    const int ntok = qg >= 2 ? ntB : ntA;
    if (ntok < 8) {   // tokens past the end of a partial window contribute nothing
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t0 = 4 * (qg & 1) + 2 * (i & 1);
        const uint32_t mask = (t0 < ntok ? 0x0000FFFFu : 0u) | (t0 + 1 < ntok ? 0xFFFF0000u : 0u);
#pragma unroll
        for (int cp = 0; cp < 4; ++cp) vh.d[cp][i] &= mask;
      }
    }
    bf16x4 pv;
#pragma unroll
    for (int j = 0; j < 4; ++j) pv[j] = (__bf16)p[j];
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      const u32x4 d = vh.d[cb >> 1];
      const uint32_t w0 = (cb & 1) ? d[2] : d[0], w1 = (cb & 1) ? d[3] : d[1];
      st.o[cb] = mfma16_bf16(pv, __builtin_bit_cast(bf16x4, make_uint2(w0, w1)), st.o[cb]);
    }
  } else {
    const bool q4 = kind == KIND_Q4;
    const u32x4 cw = vh.d[0];
    f16x4 pv;
#pragma unroll
    for (int j = 0; j < 4; ++j) pv[j] = (_Float16)p[j];
#pragma unroll
    for (int cp = 0; cp < 4; ++cp) {
      // codes of channel blocks 2 cp (elements 0..3) and 2 cp + 1 (4..7), tokens 4 qg + j
      const f16x8 c8 = q4 ? unpack_codes<4>(cw[cp], 0) : unpack_codes<2>(cw[cp >> 1], cp & 1);
      // value group cp: scales then zero points of the lane's four tokens
      // (elements copied out first: a bit cast of a vector element reads element 0)
      const u32x4 m = vh.d[1 + cp];
      const uint32_t m0 = m[0], m1 = m[1], m2 = m[2], m3 = m[3];
      const f16x2 s01 = __builtin_bit_cast(f16x2, m0), s23 = __builtin_bit_cast(f16x2, m1);
      const f16x2 z01 = __builtin_bit_cast(f16x2, m2), z23 = __builtin_bit_cast(f16x2, m3);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const f16x2 c01 = {c8[4 * e], c8[4 * e + 1]}, c23 = {c8[4 * e + 2], c8[4 * e + 3]};
        const f16x2 v01 = __builtin_elementwise_fma(s01, c01, z01);
        const f16x2 v23 = __builtin_elementwise_fma(s23, c23, z23);
        const f16x4 vv = {v01[0], v01[1], v23[0], v23[1]};
        st.o[2 * cp + e] = mfma16_f16(pv, vv, st.o[2 * cp + e]);
      }
    }
  }
  const int jc = r >> 2, h = r & 3;
  if (qg == 0 && r < 8 && h < G.gqa && (jc == 0 || pb))
    mref[(int64_t)(jc ? itB : itA) * G.H_q + g * G.gqa + h] = make_float2(st.m, lw);
  (void)ntB;
}

// End of a run: each head's two streams (O rows h and 4 + h, references and sums
// in lanes h and 4 + h) merged into O row h and lane h.
__device__ __forceinline__ void merge_streams(WaveState& st, int qg, int r) {
  float f0[4], f1[4], M[4], L[4];
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const float m0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(st.m), h));
    const float m1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(st.m), 4 + h));
    const float l0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(st.l), h));
    const float l1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(st.l), 4 + h));
    M[h] = fmaxf(m0, m1);
    f0[h] = m0 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m0 - M[h]);
    f1[h] = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - M[h]);
    L[h] = l0 * f0[h] + l1 * f1[h];
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const float fv = qg == 0 ? f0[v] : (qg == 1 ? f1[v] : 0.f);
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      const uint32_t u = __float_as_uint(st.o[cb][v] * fv);
      const auto s = __builtin_amdgcn_permlane16_swap(u, u, false, false);   // lane ^ 16
      const uint32_t s0 = s[0], s1 = s[1];
      st.o[cb][v] = __uint_as_float(s0) + __uint_as_float(s1);
    }
  }
  const int h = r & 3;
  st.m = h == 0 ? M[0] : (h == 1 ? M[1] : (h == 2 ? M[2] : M[3]));
  st.l = h == 0 ? L[0] : (h == 1 ? L[1] : (h == 2 ? L[2] : L[3]));
}

// Offset of a q*s operand entry in the per-wave staging area: the B operand of
// the QK^T MFMA, lane L = 16 q + r holding channels 8 q .. of block kb for head r.
__device__ __forceinline__ int qst_off(int hilo, int kb, int L) { return ((hilo * 4 + kb) * 64 + L) * 16; }

// QK^T and the online-softmax update of one window: probabilities in p_,
// the window's (reference, sum) pair in m_w, l_w.  The open window takes this
// step's key (and stores it into its ring slot).
// a 16-byte register of lane src
__device__ __forceinline__ u32x4 shfl16(u32x4 v, int src) {
  u32x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = (uint32_t)__shfl((int)v[i], src, 64);
  return o;
}

// QK^T of a quantized window with RoPE (keys quantized before rotation): the
// query is turned back to the window's first position, q' = R(-p0) q, and the
// dequantized keys z + s c are rotated by their offset j in the window (the
// first rows of the position table), so q' . R(j) x = q . R(p0 + j) x.  Both
// operands are split into fp16 hi + lo (three MFMAs per block: hi.hi, hi.lo,
// lo.hi), the error of the rotation in float32 stays near 2^-22.
template <int W, int NHS>
__device__ __forceinline__ void qk_rope_quant(const ItemInfo& in, const KHalf<W, true>& kh,
                                              const float (&qf)[NHS][8], uint8_t* qlds,
                                              const Geometry& G, int lane, int qg, int r,
                                              f32x4 (&acc)[W / 16]) {
  constexpr int TB = W / 16, NC = W / 16;
  const bool is4 = in.kind == KIND_Q4;
  const int gqa = G.gqa;
  uint32_t kw[4 * NC];
#pragma unroll
  for (int m = 0; m < NC; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) kw[4 * m + i] = kh.d[m][i];
  // q' = R(-p0) q: lane r holds channels 8 r .. 8 r + 7, whose partners (+-64) lane r ^ 8
  // holds; (cos, sin) of p0 for them were loaded with the window
  float cs0[16];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int i = 0; i < 4; ++i) cs0[4 * k + i] = __uint_as_float(kh.d[NC + 2 + k][i]);
  wave_sync_lds();
#pragma unroll
  for (int k = 0; k < NHS; ++k) {
    const int hh = qg + 4 * k;
    f16x8 hi8, lo8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float x = qf[k][i], y = __shfl_xor(qf[k][i], 8, 64);
      const float c = cs0[2 * i], sn = cs0[2 * i + 1];
      const float v = r < 8 ? x * c + y * sn : x * c - y * sn;
      const _Float16 h = (_Float16)v;
      hi8[i] = h;
      lo8[i] = (_Float16)(v - (float)h);
    }
    if (hh < gqa) {
      const int dst = 16 * (r & 3) + hh;   // lane of the B operand: head hh, channel group r & 3
      const int kb = r >> 2;
      *(u32x4*)(qlds + ((0 * 4 + kb) * 64 + dst) * 16) = __builtin_bit_cast(u32x4, hi8);
      *(u32x4*)(qlds + ((1 * 4 + kb) * 64 + dst) * 16) = __builtin_bit_cast(u32x4, lo8);
    }
  }
  wave_sync_lds();
  f16x8 qhi[4], qlo[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    qhi[kb] = __builtin_bit_cast(f16x8, ld16(qlds + ((0 * 4 + kb) * 64 + lane) * 16));
    qlo[kb] = __builtin_bit_cast(f16x8, ld16(qlds + ((1 * 4 + kb) * 64 + lane) * 16));
  }
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    acc[tb] = (f32x4){0.f, 0.f, 0.f, 0.f};
    const int j = 16 * tb + r;   // token offset in the window
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f16x8 ca, cb;   // codes of channels 32 kb + 8 qg + i and their partners + 64
      int ee;
      if (is4) {
        ca = unpack_codes<4>(code_word<4>(kw, tb * 4 + kb, &ee), ee);
        cb = unpack_codes<4>(code_word<4>(kw, tb * 4 + kb + 2, &ee), ee);
      } else {
        ca = unpack_codes<2>(code_word<2>(kw, tb * 4 + kb, &ee), ee);
        cb = unpack_codes<2>(code_word<2>(kw, tb * 4 + kb + 2, &ee), ee);
      }
      // scale / zero of channels 32 kb + 8 qg + i (and + 64): lane 4 kb + qg of
      // this lane's row holds channels 8 (4 kb + qg) .. + 7 in its compact registers
      const int src_a = 16 * qg + 4 * kb + qg, src_b = src_a + 8;
      const f16x8 sa = __builtin_bit_cast(f16x8, shfl16(kh.d[NC], src_a));
      const f16x8 za = __builtin_bit_cast(f16x8, shfl16(kh.d[NC + 1], src_a));
      const f16x8 sb = __builtin_bit_cast(f16x8, shfl16(kh.d[NC], src_b));
      const f16x8 zb = __builtin_bit_cast(f16x8, shfl16(kh.d[NC + 1], src_b));
      const float* cj = G.rope + 2 * ((int64_t)j * (kHeadDim / 2) + 32 * kb + 8 * qg);
      float cs[16];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const u32x4 v = ld16(cj + 4 * k);
#pragma unroll
        for (int i = 0; i < 4; ++i) cs[4 * k + i] = __uint_as_float(v[i]);
      }
      f16x8 ahi, alo, bhi, blo;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float xa = fmaf((float)sa[i], (float)ca[i], (float)za[i]);
        const float xb = fmaf((float)sb[i], (float)cb[i], (float)zb[i]);
        const float c = cs[2 * i], sn = cs[2 * i + 1];
        const float ra = xa * c - xb * sn, rb = xb * c + xa * sn;
        ahi[i] = (_Float16)ra;
        alo[i] = (_Float16)(ra - (float)ahi[i]);
        bhi[i] = (_Float16)rb;
        blo[i] = (_Float16)(rb - (float)bhi[i]);
      }
      acc[tb] = mfma_f16(ahi, qhi[kb], acc[tb]);
      acc[tb] = mfma_f16(ahi, qlo[kb], acc[tb]);
      acc[tb] = mfma_f16(alo, qhi[kb], acc[tb]);
      acc[tb] = mfma_f16(bhi, qhi[kb + 2], acc[tb]);
      acc[tb] = mfma_f16(bhi, qlo[kb + 2], acc[tb]);
      acc[tb] = mfma_f16(blo, qhi[kb + 2], acc[tb]);
    }
  }
}

template <int W, int NHS, bool ROPE>
__device__ __forceinline__ void process_k(const ItemInfo& in, KHalf<W, ROPE>& kh, WaveState& st,
                                          const bf16x8 (&qop)[4], const float (&qf)[NHS][8],
                                          uint8_t* qlds, const AttnArgs& a, int b, int g, int lane,
                                          int qg, int r, float (&p_)[row_tiles<W>()][4], float* m_w,
                                          float* l_w) {
  constexpr int TB = row_tiles<W>();
  const Geometry& G = a.g;
  const int gqa = G.gqa;
  const int ntok = in.ntok;
  f32x4 acc[TB];
  if (in.kind == KIND_BF16) {
    if (in.open) {   // the token appended this step: use it from the input and store it
      const int pos = ntok - 1;
      const uint16_t* kn = a.k_new + ((int64_t)b * G.H_kv + g) * kHeadDim;
      uint8_t* pw = const_cast<uint8_t*>(in.p);
      // keys: the lanes whose row is token pos take the new key (selects, no
      // conditional writes into the operand registers)
      const bool krow = r == (pos & 15);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const u32x4 v = ld16(kn + 32 * kb + 8 * qg);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          const bool sel = krow && tb == (pos >> 4);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t old = kh.d[tb * 4 + kb][i], nv = v[i];
            kh.d[tb * 4 + kb][i] = sel ? nv : old;
          }
          if (sel) {
            const int64_t off = W == 8 ? (int64_t)((kb * 4 + qg) * 8 + r) * 16
                                       : (int64_t)((tb * 4 + kb) * 64 + lane) * 16;
            *(u32x4*)(pw + off) = v;
          }
        }
      }
    }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      acc[tb] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        acc[tb] = mfma_bf16(__builtin_bit_cast(bf16x8, kh.d[tb * 4 + kb]), qop[kb], acc[tb]);
    }
    softmax_window<TB, NHS>(acc, 0.f, ntok, G.scale_log2, qg, st, p_, m_w, l_w);
  } else if constexpr (ROPE) {
    qk_rope_quant<W, NHS>(in, kh, qf, qlds, G, lane, qg, r, acc);
    softmax_window<TB, NHS>(acc, 0.f, ntok, G.scale_log2, qg, st, p_, m_w, l_w);
  } else {
    // ---- quantized window: int4 or int2 codes ----
    constexpr int NC = key_code_regs<W>();
    const bool is4 = in.kind == KIND_Q4;
    uint32_t kw[4 * NC];
#pragma unroll
    for (int m = 0; m < NC; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) kw[4 * m + i] = kh.d[m][i];
    const u32x4 ks8 = kh.d[NC], kz8 = kh.d[NC + 1];

    f16x8 qhi[4], qlo[4];
    float bias = 0.f;
    if constexpr (use_reg_qs<W, NHS, ROPE>()) {
      // q*s of column r & 3, channels 32 kb + 8 q + i of block kb = r >> 2, split
      // into exact fp16 hi + lo; the column's other blocks from lanes r + 4j
      // (block kb = r >> 2 of the query picked with masks: a select over the array
      // would become an indexed access, which the compiler puts in scratch)
      const int kbl = r >> 2;
      u32x4 qb = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const uint32_t m = kbl == kb ? ~0u : 0u;
        const u32x4 v = __builtin_bit_cast(u32x4, qop[kb]);
#pragma unroll
        for (int i = 0; i < 4; ++i) qb[i] |= v[i] & m;
      }
      float bsum = 0.f;
      f16x8 hi8, lo8;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float qv = __uint_as_float((i & 1) ? (qb[i >> 1] & 0xFFFF0000u) : (qb[i >> 1] << 16));
        const float sv = (float)__builtin_bit_cast(_Float16, (uint16_t)(ks8[i >> 1] >> (16 * (i & 1))));
        const float zv = (float)__builtin_bit_cast(_Float16, (uint16_t)(kz8[i >> 1] >> (16 * (i & 1))));
        const float qs = qv * sv;   // exact: 8-bit x 11-bit significands
        const _Float16 h = (_Float16)qs;
        hi8[i] = h;
        lo8[i] = (_Float16)(qs - (float)h);
        bsum = fmaf(qv, zv, bsum);
      }
      const u32x4 mh = __builtin_bit_cast(u32x4, hi8), ml = __builtin_bit_cast(u32x4, lo8);
      qhi[0] = hi8;
      qlo[0] = lo8;
      qhi[1] = __builtin_bit_cast(f16x8, row_ror<12>(mh));   // lane r + 4
      qlo[1] = __builtin_bit_cast(f16x8, row_ror<12>(ml));
      qhi[2] = __builtin_bit_cast(f16x8, row_ror<8>(mh));    // lane r + 8
      qlo[2] = __builtin_bit_cast(f16x8, row_ror<8>(ml));
      qhi[3] = __builtin_bit_cast(f16x8, row_ror<4>(mh));    // lane r + 12
      qlo[3] = __builtin_bit_cast(f16x8, row_ror<4>(ml));
      // q . z of the column: its four blocks (lanes r + 4j), then the four lane groups
      bsum += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(bsum), 0x128, 0xF, 0xF, false));
      bsum += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(bsum), 0x124, 0xF, 0xF, false));
      bias = rows_sum(bsum);
    } else {
    // q*s split into exact fp16 hi + lo, written as the B operand layout
    float bias_k[NHS];
    wave_sync_lds();
#pragma unroll
    for (int k = 0; k < NHS; ++k) {
      const int hh = qg + 4 * k;
      float bsum = 0.f;
      f16x8 hi8, lo8;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint16_t sbits = (uint16_t)(ks8[i >> 1] >> (16 * (i & 1)));
        const uint16_t zbits = (uint16_t)(kz8[i >> 1] >> (16 * (i & 1)));
        const float sv = (float)__builtin_bit_cast(_Float16, sbits);
        const float zv = (float)__builtin_bit_cast(_Float16, zbits);
        const float qs = qf[k][i] * sv;   // exact: 8-bit x 11-bit significands
        const _Float16 h = (_Float16)qs;
        hi8[i] = h;
        lo8[i] = (_Float16)(qs - (float)h);
        bsum = fmaf(qf[k][i], zv, bsum);
      }
      if (hh < gqa) {
        const int dst = 16 * (r & 3) + hh;   // lane of the B operand: head hh, channel group r & 3
        const int kb = r >> 2;
        *(u32x4*)(qlds + qst_off(0, kb, dst)) = __builtin_bit_cast(u32x4, hi8);
        *(u32x4*)(qlds + qst_off(1, kb, dst)) = __builtin_bit_cast(u32x4, lo8);
      }
      bias_k[k] = row16_sum(bsum);   // q . z of head qg + 4k (same value in all 16 lanes)
    }
#pragma unroll
    for (int k = 0; k < NHS; ++k) {
      const float t = __shfl(bias_k[k], 16 * (r & 3));
      if ((r >> 2) == k) bias = t;
    }
    wave_sync_lds();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      qhi[kb] = __builtin_bit_cast(f16x8, ld16(qlds + qst_off(0, kb, lane)));
      qlo[kb] = __builtin_bit_cast(f16x8, ld16(qlds + qst_off(1, kb, lane)));
    }
    }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      acc[tb] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int e = tb * 4 + kb;
        int ee;
        f16x8 cv;
        if (is4) {
          uint32_t w = code_word<4>(kw, e, &ee);
          cv = unpack_codes<4>(w, ee);
        } else {
          uint32_t w = code_word<2>(kw, e, &ee);
          cv = unpack_codes<2>(w, ee);
        }
        acc[tb] = mfma_f16(cv, qhi[kb], acc[tb]);
        acc[tb] = mfma_f16(cv, qlo[kb], acc[tb]);
      }
    }
    softmax_window<TB, NHS>(acc, bias, ntok, G.scale_log2, qg, st, p_, m_w, l_w);
  }
}

// P.V of an 8-token window: 16x16x16 MFMAs whose A operand is the lane's four
// probabilities as the QK^T accumulator left them (head r, tokens 4 qg .. + 3)
// and whose B operand holds the window's values in lanes qg < 2; the other
// token columns carry zero probabilities and zero values.  The open window
// takes this step's value (and stores it); tokens past the end of a partial
// window contribute nothing.
template <int NHS>
__device__ __forceinline__ void process_v8(const ItemInfo& in, VHalf<8>& vh, WaveState& st,
                                           const float (&p_)[1][4], float m_w, float l_w,
                                           const AttnArgs& a, int b, int g, int qg, int r,
                                           float2* mref) {
  const Geometry& G = a.g;
  const int gqa = G.gqa;
  const int ntok = in.ntok;
  if (in.kind == KIND_BF16) {
    if (in.open) {
      const int pos = ntok - 1;   // token 4 qp + jp: element jp of lanes qg == qp
      const int qp = pos >> 2, jp = pos & 3;
      const uint16_t* vn = a.v_new + ((int64_t)b * G.H_kv + g) * kHeadDim;
      uint8_t* pw = const_cast<uint8_t*>(in.p);
      const bool vgrp = qg == qp;
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) {
        const uint32_t val = vn[16 * cb + r];
        if (vgrp) *(uint16_t*)(pw + v_elem_off(8, pos, 16 * cb + r)) = (uint16_t)val;
        const int wi = (cb & 1) * 2 + (jp >> 1);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t wv = vh.d[cb >> 1][i];
          const uint32_t lo = (wv & 0xFFFF0000u) | val, hi = (wv & 0x0000FFFFu) | (val << 16);
          vh.d[cb >> 1][i] = (vgrp && i == wi) ? ((jp & 1) ? hi : lo) : wv;
        }
      }
    }
    if (ntok < 8) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t0 = 4 * qg + 2 * (i & 1);
        const uint32_t mask = (t0 < ntok ? 0x0000FFFFu : 0u) | (t0 + 1 < ntok ? 0xFFFF0000u : 0u);
#pragma unroll
        for (int cp = 0; cp < 4; ++cp) vh.d[cp][i] &= mask;
      }
    }
    bf16x4 pv;
#pragma unroll
    for (int j = 0; j < 4; ++j) pv[j] = (__bf16)p_[0][j];
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      const u32x4 d = vh.d[cb >> 1];
      const uint32_t w0 = (cb & 1) ? d[2] : d[0], w1 = (cb & 1) ? d[3] : d[1];
      const bf16x4 vb = __builtin_bit_cast(bf16x4, make_uint2(w0, w1));
      st.o[cb] = mfma16_bf16(pv, vb, st.o[cb]);
    }
  } else {
    const bool is4 = in.kind == KIND_Q4;
    const u32x4 cw = vh.d[0];
    f16x4 pv;
#pragma unroll
    for (int j = 0; j < 4; ++j) pv[j] = (_Float16)p_[0][j];
#pragma unroll
    for (int cp = 0; cp < 4; ++cp) {
      // codes of channel blocks 2 cp (elements 0..3) and 2 cp + 1 (4..7), tokens 4 qg + j
      const uint32_t w4 = cw[cp], w2 = cw[cp >> 1];
      const f16x8 c8 = is4 ? unpack_codes<4>(w4, 0) : unpack_codes<2>(w2, cp & 1);
      // value group cp: scales then zero points of the lane's four tokens
      const u32x4 m = vh.d[1 + cp];
      const uint32_t m0 = m[0], m1 = m[1], m2 = m[2], m3 = m[3];
      const f16x2 s01 = __builtin_bit_cast(f16x2, m0), s23 = __builtin_bit_cast(f16x2, m1);
      const f16x2 z01 = __builtin_bit_cast(f16x2, m2), z23 = __builtin_bit_cast(f16x2, m3);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const f16x2 c01 = {c8[4 * e], c8[4 * e + 1]}, c23 = {c8[4 * e + 2], c8[4 * e + 3]};
        const f16x2 v01 = __builtin_elementwise_fma(s01, c01, z01);
        const f16x2 v23 = __builtin_elementwise_fma(s23, c23, z23);
        const f16x4 vv = {v01[0], v01[1], v23[0], v23[1]};
        st.o[2 * cp + e] = mfma16_f16(pv, vv, st.o[2 * cp + e]);
      }
    }
  }
  if (qg == 0 && r < gqa) mref[(int64_t)in.it * G.H_q + g * gqa + r] = make_float2(m_w, l_w);
}

// P.V of one window into the running output, then the window's statistics.
// The open window takes this step's value (and stores it); tokens past the end
// of a partial window contribute nothing.
template <int W, int NHS>
__device__ __forceinline__ void process_v(const ItemInfo& in, VHalf<W>& vh, WaveState& st,
                                          const float (&p_)[row_tiles<W>()][4], float m_w, float l_w,
                                          const AttnArgs& a, int b, int g, int qg, int r,
                                          float2* mref) {
  if constexpr (W == 8) {
    process_v8<NHS>(in, vh, st, p_, m_w, l_w, a, b, g, qg, r, mref);
    return;
  }
  constexpr int KT = W / 32;
  const Geometry& G = a.g;
  const int gqa = G.gqa;
  const int ntok = in.ntok;
  if (in.kind == KIND_BF16) {
    if (ntok < W || in.open) {
      const int pos = ntok - 1;
      if (in.open) {
        const uint16_t* vn = a.v_new + ((int64_t)b * G.H_kv + g) * kHeadDim;
        uint8_t* pw = const_cast<uint8_t*>(in.p);
        // values: element j of the lanes in group qp holds token pos
        int ktp, qp, jp;
        v_tok_pos(pos, &ktp, &qp, &jp);
        const bool vgrp = qg == qp;
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) {
          const uint32_t val = vn[16 * cb + r];
          if (vgrp) *(uint16_t*)(pw + v_elem_off(W, pos, 16 * cb + r)) = (uint16_t)val;
#pragma unroll
          for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const bool here = vgrp && kt == ktp && (jp >> 1) == i;
              const uint32_t wv = vh.d[kt * 8 + cb][i];
              const uint32_t lo = (wv & 0xFFFF0000u) | val, hi = (wv & 0x0000FFFFu) | (val << 16);
              vh.d[kt * 8 + cb][i] = here ? ((jp & 1) ? hi : lo) : wv;
            }
        }
      }
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool lo_ok = v_tok(kt, qg, 2 * i) < ntok, hi_ok = v_tok(kt, qg, 2 * i + 1) < ntok;
          const uint32_t mask = (lo_ok ? 0x0000FFFFu : 0u) | (hi_ok ? 0xFFFF0000u : 0u);
#pragma unroll
          for (int cb = 0; cb < 8; ++cb) vh.d[kt * 8 + cb][i] &= mask;
        }
    }
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      bf16x8 pv;
#pragma unroll
      for (int j = 0; j < 8; ++j) pv[j] = (__bf16)p_[2 * kt + (j >> 2)][j & 3];
#pragma unroll
      for (int cb = 0; cb < 8; ++cb)
        st.o[cb] = mfma_bf16(pv, __builtin_bit_cast(bf16x8, vh.d[kt * 8 + cb]), st.o[cb]);
    }
  } else {
    constexpr int NC = key_code_regs<W>();   // (8-token windows take process_v8)
    constexpr int NG = kHeadDim / W;
    const bool is4 = in.kind == KIND_Q4;
    uint32_t vw[4 * NC];
#pragma unroll
    for (int m = 0; m < NC; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) vw[4 * m + i] = vh.d[m][i];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      f16x8 pv;
#pragma unroll
      for (int j = 0; j < 8; ++j) pv[j] = (_Float16)p_[2 * kt + (j >> 2)][j & 3];
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) {
        const int e = kt * 8 + cb;
        const int vg = (16 * cb) / W;
        int ee;
        f16x8 cv;
        if (is4) {
          uint32_t w = code_word<4>(vw, e, &ee);
          cv = unpack_codes<4>(w, ee);
        } else {
          uint32_t w = code_word<2>(vw, e, &ee);
          cv = unpack_codes<2>(w, ee);
        }
        const u32x4 sv4 = vh.d[NC + (kt * NG + vg) * 2];
        const u32x4 zv4 = vh.d[NC + 1 + (kt * NG + vg) * 2];
        f16x8 vv;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // vector elements go through scalars: bit-casting an element of an
          // ext_vector directly reads element 0 with this compiler
          const uint32_t si = sv4[i], zi = zv4[i];
          f16x2 c2 = {cv[2 * i], cv[2 * i + 1]};
          f16x2 r2 = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, si), c2,
                                               __builtin_bit_cast(f16x2, zi));
          vv[2 * i] = r2[0];
          vv[2 * i + 1] = r2[1];
        }
        st.o[cb] = mfma_f16(pv, vv, st.o[cb]);
      }
    }
  }
  if (qg == 0 && r < gqa) mref[(int64_t)in.it * G.H_q + g * gqa + r] = make_float2(m_w, l_w);
}

constexpr int kAttnSmemFixed = 4 * 16 * 130 * 4;   // q*s staging per wave / end-of-split merge
// Dynamic LDS of a workgroup before its live-list entries: the q*s staging of
// the four waves (compact when the LDS slots are used: the slots are a static
// array of their own, which also holds the end-of-split merge; otherwise the
// merge reuses the staging area)
template <int W, int NHS, bool ROPE>
constexpr int attn_smem_fixed() { return use_slot<W, NHS, ROPE>() ? 0 : kAttnSmemFixed; }

// MINB workgroups of four waves per compute unit: at most 512 / MINB VGPRs per lane
template <int W, int NHS, int MINB, bool ROPE>
__global__ __launch_bounds__(kAttnThreads, MINB) void k_attend(AttnArgs a) {
  const Geometry& G = a.g;
  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, qg = lane >> 4;
  const int gqa = G.gqa;

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr bool SLOT = use_slot<W, NHS, ROPE>();
  // q*s staging: [hi/lo][kb][lane] x 16 B (pairs of 8-token windows form q*s in registers)
  uint8_t* qlds = smem + wave * 8192;
  uint8_t* mo_base = smem;   // end-of-split merge of the four waves
  int32_t* s_ref = (int32_t*)(smem + attn_smem_fixed<W, NHS, ROPE>());   // live-list entries

  uint8_t* ub = a.base + (int64_t)b * a.L.unit_bytes;
  const int32_t* counts = (const int32_t*)(ub + a.L.counts);
  const int32_t* icost = (const int32_t*)(ub + a.L.item_cost);
  const int32_t* iref = (const int32_t*)(ub + a.L.item_ref);
  const int32_t* iwin_l = (const int32_t*)(ub + a.L.item_win);
  float2* mref = (float2*)(ub + a.L.mref);

  // ---- one round of loads: list length and cost, the first 1024 entries of the
  // live list with their cost prefixes (and the previous entry's), queries ----
  const int n_fq = __builtin_amdgcn_readfirstlane(counts[CNT_ITEMS]);
  const int base_cost = __builtin_amdgcn_readfirstlane(counts[CNT_COST]);
  // the re-rank kernel's split plans (first item, end item, first refs): this
  // wave's record in both slots, then the one whose step range holds T
  static_assert(kPlanSlots == 2 && kPlanRec == 8, "plan record: first, end, 6 refs");
  const int u_rec = s * 4 + __builtin_amdgcn_readfirstlane(wave);
  const int32_t* prec0 = (const int32_t*)(ub + a.L.plan) + u_rec * kPlanRec;
  const int32_t* prec1 = prec0 + 4 * G.n_split * kPlanRec;
  int ptag[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) ptag[j] = __builtin_amdgcn_readfirstlane(counts[CNT_PLAN_T0 + j]);
  const int rec0 = lane < kPlanRec ? prec0[lane] : 0;   // lane k: record word k
  const int rec1 = lane < kPlanRec ? prec1[lane] : 0;
  const bool in0 = ptag[0] <= a.T && a.T <= ptag[1];
  const bool plan_ok = in0 || (ptag[2] <= a.T && a.T <= ptag[3]);
  const int rec = in0 ? rec0 : rec1;
  const int p_first = __builtin_amdgcn_readlane(rec, 0);
  const int p_last = __builtin_amdgcn_readlane(rec, 1);
  int32_t lc[4], lp[4], lr[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int i = tid + k * kAttnThreads;
    lc[k] = i <= G.max_fq ? icost[i] : 0;
    lp[k] = i >= 1 && i <= G.max_fq + 1 ? icost[i - 1] : -1;
    lr[k] = i < G.max_fq ? iref[i] : 0;
  }
  const uint16_t* qbase = a.q + ((int64_t)b * G.H_q + (int64_t)g * gqa) * kHeadDim;
  bf16x8 qop[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    // column r: head r (pairs of 8-token windows: head r & 3 of column block
    // (r >> 2) & 1; columns 8..15 repeat 0..7 and are masked)
    const int hc = (SLOT || use_reg_qs<W, NHS, ROPE>()) ? (r & 3) : r;
    u32x4 v = {0, 0, 0, 0};
    if (hc < gqa) v = ld16(qbase + hc * kHeadDim + 32 * kb + 8 * qg);
    qop[kb] = __builtin_bit_cast(bf16x8, v);
  }
  float qf[NHS][8];   // compact: head qg + 4k, channels 8r .. 8r + 7
#pragma unroll
  for (int k = 0; k < NHS; ++k) {
    const int hh = qg + 4 * k;
    u32x4 v = {0, 0, 0, 0};
    if (hh < gqa) v = ld16(qbase + hh * kHeadDim + 8 * r);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      qf[k][2 * i] = __uint_as_float(v[i] << 16);
      qf[k][2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
    }
  }
  // zero this lane's q*s operand slots (padded heads keep zeros)
  if constexpr (!SLOT && !use_reg_qs<W, NHS, ROPE>()) {
#pragma unroll
    for (int i = 0; i < 8; ++i) *(u32x4*)(qlds + (i * 64 + lane) * 16) = (u32x4){0, 0, 0, 0};
  }

  // ---- this wave's item range: from the plan, else computed here ----
  const int n_extra = a.n_ring + a.n_sink_items;
  int first, last;
  if (plan_ok) {
    first = p_first;
    last = p_last;
  } else {
    // ---- this split's item range (equal estimated cost) ----
    // Items: the live list, then the recent-region and sink windows (cost cF each).
    // The split is cut into 4 equal-cost parts, one per wave: part u = 4s + w holds
    // the items whose start cost lies in [ceil(u total / 4S), ceil((u + 1) total / 4S)).
    // s_range[j] = first item whose start cost reaches the j-th cut of this split:
    // start costs increase strictly, so the item with start(i - 1) < cut <= start(i)
    // is unique, and cuts beyond the last item's start are set by that item.
    // Costs are small integers (at most 32 per window, under 2^13 windows), so every
    // prefix and cut fits in 32 bits; the cuts are uniform (scalar unit).
    const int n_all = n_fq + n_extra;
    const int cF = G.cost_bf16;
    const int total = base_cost + n_extra * cF;
    const int S = G.n_split;
    __shared__ int s_range[5];
    const uint32_t S4 = 4u * (uint32_t)S;
    int cut[5];
#pragma unroll
    for (int j = 0; j < 5; ++j) cut[j] = (int)(((4u * (uint32_t)s + j) * (uint32_t)total + S4 - 1) / S4);
    auto place = [&](int i, int c0, int c1) {
      // bit j: cut j falls in (c0, c1] (or, for the last item, beyond it)
      uint32_t m = 0, m_end = 0;
#pragma unroll
      for (int j = 0; j < 5; ++j) {
        m |= (c1 >= cut[j] && c0 < cut[j]) ? 1u << j : 0u;
        m_end |= cut[j] > c1 ? 1u << j : 0u;
      }
      if (i == n_all - 1) {
        for (uint32_t e = m_end; e; e &= e - 1) s_range[__builtin_ctz(e)] = n_all;
      }
      for (; m; m &= m - 1) s_range[__builtin_ctz(m)] = i;
    };
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (k * kAttnThreads >= n_all) break;   // uniform
      const int i = tid + k * kAttnThreads;
      if (i < n_fq) s_ref[i] = lr[k];
      if (i < n_all) {
        const int c1 = i <= n_fq ? lc[k] : base_cost + (i - n_fq) * cF;
        const int c0 = i == 0 ? -1 : (i - 1 <= n_fq ? lp[k] : base_cost + (i - 1 - n_fq) * cF);
        place(i, c0, c1);
      }
    }
    // long lists: rounds of four entries per thread, all loads of a round first
    for (int i0 = 4 * kAttnThreads; i0 < n_all; i0 += 4 * kAttnThreads) {
      int xc[4], xp[4], xr[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int i = i0 + tid + k * kAttnThreads;
        xc[k] = i <= n_fq ? icost[i] : 0;
        xp[k] = i - 1 <= n_fq ? icost[i - 1] : 0;
        xr[k] = i < n_fq ? iref[i] : 0;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int i = i0 + tid + k * kAttnThreads;
        if (i >= n_all) break;
        if (i < n_fq) s_ref[i] = xr[k];
        const int c1 = i <= n_fq ? xc[k] : base_cost + (i - n_fq) * cF;
        const int c0 = i - 1 <= n_fq ? xp[k] : base_cost + (i - 1 - n_fq) * cF;
        place(i, c0, c1);
      }
    }
    if (n_all == 0 && tid < 5) s_range[tid] = 0;
    __syncthreads();

    // (the 8-token pair loop wants its run bounds in scalar registers; for the
    // others that costs registers in the loop)
    first = SLOT ? __builtin_amdgcn_readfirstlane(s_range[wave]) : s_range[wave];
    last = SLOT ? __builtin_amdgcn_readfirstlane(s_range[wave + 1]) : s_range[wave + 1];
  }

  // plan path: list refs of a run past the plan record's first ones, one per lane
  int run_ref = 0;
  if (plan_ok && last - first > kPlanRefs) {   // uniform
    const int i = first + kPlanRefs + lane;
    run_ref = i < last && i < n_fq ? iref[i] : 0;
  }

  WaveState st;
  st.m = -INFINITY;
  st.l = 0.f;
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) st.o[cb] = (f32x4){0.f, 0.f, 0.f, 0.f};

  const int w_open = (a.T - 1 - G.sink) / W;
  uint8_t* fpool = ub + a.L.fpool;
  uint8_t* qpool = ub + a.L.qpool;
  uint8_t* ring = ub + a.L.ring;
  uint8_t* sinkp = ub + a.L.sinkp;
  auto info = [&](int it) {
    ItemInfo in;
    in.it = it;
    in.kind = KIND_BF16;
    in.ntok = W;
    in.open = false;
    in.win = -1;
    if (it < n_fq) {
      if constexpr (ROPE) in.win = iwin_l[it];
      int32_t ref;
      if (plan_ok) {
        const int k = it - first;
        ref = k < kPlanRefs        ? __builtin_amdgcn_readlane(rec, 2 + k)
              : k < kPlanRefs + 64 ? __builtin_amdgcn_readlane(run_ref, k - kPlanRefs)
                                   : iref[it];
      } else {
        ref = s_ref[it];
      }
      ref = __builtin_amdgcn_readfirstlane(ref);   // one item per wave: scalar branches on its kind
      in.kind = ref >> 28;
      const int64_t slot = ref & 0x0FFFFFFF;
      in.p = in.kind == KIND_BF16 ? fpool + slot * G.fslot_bytes + g * G.fhead_bytes
                                  : qpool + slot * G.qslot_bytes + g * G.qrec_bytes;
    } else if (it < n_fq + a.n_ring) {
      const int w = a.ring_w0 + (it - n_fq);
      in.p = ring + (int64_t)(w % G.NR) * G.fslot_bytes + g * G.fhead_bytes;
      in.ntok = min(W, a.T - (G.sink + w * W));
      in.open = (w == w_open);
    } else {
      const int j = it - n_fq - a.n_ring;
      in.p = sinkp + (int64_t)j * G.fslot_bytes + g * G.fhead_bytes;
      in.ntok = min(W, G.sink - j * W);
    }
    return in;
  };

  // ---- window loop: this wave's contiguous run of windows ----
  constexpr int TB = row_tiles<W>();
  KHalf<W, ROPE> KA;
  VHalf<W> V;
  float p_[TB][4];
  float m_w, l_w;
  if constexpr (SLOT) {
    // pairs of windows through the wave's LDS slot: wait for the pair, gather its
    // operands, start the next pair's loads into the slot, then compute
    __shared__ __attribute__((aligned(16))) uint8_t s_slots[4 * 2 * kPairSlot];
    uint8_t* slot = s_slots + wave * 2 * kPairSlot;
    mo_base = s_slots;
    // the pair starting at item i: its second item, and whether it has one
    auto pair_at = [&](int i, ItemInfo& x, ItemInfo& y) {
      x = info(i);
      y = info(i + 1 < last ? i + 1 : i);
      return i + 1 < last && y.kind == x.kind;
    };
    if (first < last) {
      ItemInfo ia, ib;
      bool pb = pair_at(first, ia, ib);
      issue_record(ia, slot, lane, G);
      if (pb) issue_record(ib, slot + kPairSlot, lane, G);
      f16x8 qhi[4], qlo[4];
      float bias;
      for (int it = first; it < last;) {
        const int nxt = it + (pb ? 2 : 1);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        read_pair(ia.kind, pb, slot, KA, V, qhi, qlo, &bias, qop, r, qg, G);
        wave_sync_lds();
        if (ia.open) patch_open8(ia, 0, KA, V, a, b, g, qg, r);
        if (pb && ib.open) patch_open8(ib, 1, KA, V, a, b, g, qg, r);
        ItemInfo na, nb;
        const bool has = nxt < last;
        const bool npb = pair_at(has ? nxt : it, na, nb) && has;
        if (has) {
          issue_record(na, slot, lane, G);
          if (npb) issue_record(nb, slot + kPairSlot, lane, G);
        }
        __builtin_amdgcn_sched_barrier(0);
        float lw;
        pair_k(ia.kind, pb, ia.ntok, ib.ntok, KA, qop, qhi, qlo, bias, G.scale_log2, qg, r, st, p_[0], &lw);
        pair_v(ia.kind, pb, ia.it, ib.it, ia.ntok, ib.ntok, V, st, p_[0], lw, a, g, qg, r, mref);
        ia = na;
        ib = nb;
        pb = npb;
        it = nxt;
      }
    }
    merge_streams(st, qg, r);
  } else {
    for (int it = first; it < last; ++it) {
      const ItemInfo ia = info(it);
      fetch_k<W, ROPE, use_reg_qs<W, NHS, ROPE>()>(ia, KA, lane, r, G);
      fetch_v<W>(ia, V, lane, qg, G);
      process_k<W, NHS, ROPE>(ia, KA, st, qop, qf, qlds, a, b, g, lane, qg, r, p_, &m_w, &l_w);
      process_v<W, NHS>(ia, V, st, p_, m_w, l_w, a, b, g, qg, r, mref);
    }
  }

  // ---- merge the 4 waves of this split in LDS, write the split partial ----
  if constexpr (SLOT) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the last slot loads
  __syncthreads();
  constexpr int MH = SLOT ? 4 : 16;   // heads per wave in the merge buffer (gqa <= MH)
  float* mo = (float*)mo_base;        // [wave][head < MH][130]
  if (qg == 0 && r < gqa) {
    mo[(wave * MH + r) * 130 + 128] = st.m;
    mo[(wave * MH + r) * 130 + 129] = st.l;
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int row = 4 * qg + v;
    if (row < gqa) {
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) mo[(wave * MH + row) * 130 + 16 * cb + r] = st.o[cb][v];
    }
  }
  __syncthreads();
  float* part = (float*)(ub + a.L.partial);
  float2* pml = (float2*)(ub + a.L.pml);
  for (int idx = tid; idx < gqa * kHeadDim; idx += kAttnThreads) {
    const int h = idx >> 7, c = idx & 127;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, mo[(w * MH + h) * 130 + 128]);
    float o = 0.f, L = 0.f;
    if (M > -INFINITY) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float mw = mo[(w * MH + h) * 130 + 128];
        if (mw > -INFINITY) {
          const float f = __builtin_amdgcn_exp2f(mw - M);
          o += mo[(w * MH + h) * 130 + c] * f;
          L += mo[(w * MH + h) * 130 + 129] * f;
        }
      }
    }
    const int64_t row = (int64_t)(g * gqa + h) * G.n_split + s;
    part[row * kHeadDim + c] = o;
    if (c == 0) pml[row] = make_float2(M, L);
  }
}

// Split merge and window-score accumulation.
//
// Output blocks (one per query head): M = max_s m_s, L = sum_s l_s 2^(m_s - M),
// out = sum_s O_s 2^(m_s - M) / L.  Mass blocks (a few live windows each, one
// thread per (window, head)): mass_h(w) = 2^(m_w - M_h) l_w / L_h, summed over
// the query heads of each KV group, then over the groups, / H_q, added to the
// window's cumulative score.  Every thread issues all of its global loads in
// one round; the reductions run in a fixed order, so results do not depend
// on timing.
constexpr int kMergeThreads = 256;
constexpr int kSplitGroups = 8;                     // split rows handled in parallel per output block

// NSPT: split rows one output-block thread reads (>= S / 8)
// Score update of the merge: attention masses (cumulative or decayed), the
// attention p-norm, or key norms (separate instantiations, so the default one
// carries no code of the others)
enum MergeScore { kScoreMass = 0, kScorePNorm = 1, kScoreKeyNorm = 2 };

template <int NSPT, int MS>
__global__ __launch_bounds__(kMergeThreads) void k_merge(AttnArgs a) {
  const Geometry& G = a.g;
  const int blk = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  uint8_t* ub = a.base + (int64_t)b * a.L.unit_bytes;
  const int32_t* counts = (const int32_t*)(ub + a.L.counts);
  const float* part = (const float*)(ub + a.L.partial);
  const float2* pml = (const float2*)(ub + a.L.pml);
  const int S = G.n_split;
  const int nh = G.H_q;
  __shared__ float4 sred[kSplitGroups][kHeadDim / 4];
  __shared__ float sml[2][kSplitGroups];
  __shared__ float sM[64], sL[64];
  __shared__ float smass[kMergeThreads];
  __shared__ float skn[kMergeThreads];

  if (blk < nh) {
    // ---- output of head h: thread (c4, grp) owns channels 4c4..4c4+3 of splits grp + 8i ----
    const int h = blk;
    const int c4 = tid & 31, grp = tid >> 5;
    float4 o[NSPT];
    float2 ml[NSPT];
#pragma unroll
    for (int i = 0; i < NSPT; ++i) {
      const int sp = grp + kSplitGroups * i;
      const bool ok = sp < S;
      o[i] = ok ? *(const float4*)(part + ((int64_t)h * S + sp) * kHeadDim + 4 * c4)
                : make_float4(0.f, 0.f, 0.f, 0.f);
      ml[i] = ok ? pml[(int64_t)h * S + sp] : make_float2(-INFINITY, 0.f);
    }
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < NSPT; ++i) m = fmaxf(m, ml[i].x);
    if (c4 == 0) sml[0][grp] = m;
    __syncthreads();
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < kSplitGroups; ++q) M = fmaxf(M, sml[0][q]);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    float lsum = 0.f;
    if (M > -INFINITY) {
#pragma unroll
      for (int i = 0; i < NSPT; ++i) {
        const float f = ml[i].x > -INFINITY ? __builtin_amdgcn_exp2f(ml[i].x - M) : 0.f;
        acc.x += f * o[i].x;
        acc.y += f * o[i].y;
        acc.z += f * o[i].z;
        acc.w += f * o[i].w;
        lsum += f * ml[i].y;
      }
    }
    sred[grp][c4] = acc;
    if (c4 == 0) sml[1][grp] = lsum;
    __syncthreads();
    if (tid < kHeadDim / 4) {
      float4 out = make_float4(0.f, 0.f, 0.f, 0.f);
      float L = 0.f;
#pragma unroll
      for (int q = 0; q < kSplitGroups; ++q) {
        const float4 x = sred[q][tid];
        out.x += x.x;
        out.y += x.y;
        out.z += x.z;
        out.w += x.w;
        L += sml[1][q];
      }
      const float inv = L > 0.f ? 1.f / L : 0.f;
      const float v[4] = {out.x * inv, out.y * inv, out.z * inv, out.w * inv};
      const int64_t oi = ((int64_t)b * nh + h) * kHeadDim + 4 * tid;
      if (G.out_bf16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) ((uint16_t*)a.out)[oi + e] = f32_to_bf16_rne(v[e]);
      } else {
        *(float4*)((float*)a.out + oi) = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
    return;
  }

  // ---- mass blocks: thread (li, hh) = (item of the block, query head) ----
  const int per_blk = kMergeThreads / nh;
  const int li = tid / nh, hh = tid % nh;
  const int pos = (blk - nh) * per_blk + li;
  const bool in_blk = li < per_blk;
  // one round: this item's window statistics, list entry and score, all split statistics
  const int n_fq = counts[CNT_ITEMS];
  const float2* __restrict__ mref = (const float2*)(ub + a.L.mref);
  const int32_t* __restrict__ iwin = (const int32_t*)(ub + a.L.item_win);
  float* iscore = (float*)(ub + a.L.item_score);
  const bool maybe = in_blk && pos < G.max_items;
  const float2 mr = maybe ? mref[(int64_t)pos * nh + hh] : make_float2(-INFINITY, 0.f);
  const int wl = (maybe && hh == 0) ? iwin[min(pos, G.max_fq)] : -1;   // used when pos < n_fq
  const float old_score = (maybe && hh == 0) ? iscore[pos] : 0.f;
  // M_h, L_h: P consecutive threads per head (P a power of two, P * H_q <= 256,
  // P <= 64 so that the P threads of a head sit in one wave), thread j folds
  // splits j, j + P, j + 2P, ... (consecutive threads read consecutive rows),
  // then a butterfly over the P lanes combines the (max, sum) pairs
  int P = 1;
  while (2 * P * nh <= kMergeThreads && P < 64) P *= 2;
  const int C = (S + P - 1) / P;
  // C <= 32: with P = 64, S <= 256 splits; otherwise P * H_q > 128 and S * H_q <= 4096
  constexpr int kMaxC = 32;
  {
    const int h = tid / P, j = tid % P;
    const bool hv = h < nh;
    float2 st[kMaxC];
#pragma unroll
    for (int i = 0; i < kMaxC; ++i) {
      const int sp = j + P * i;
      st[i] = (hv && i < C && sp < S) ? pml[(int64_t)h * S + sp] : make_float2(-INFINITY, 0.f);
    }
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < kMaxC; ++i) m = fmaxf(m, st[i].x);
    float l = 0.f;
    if (m > -INFINITY) {
#pragma unroll
      for (int i = 0; i < kMaxC; ++i)
        if (st[i].x > -INFINITY) l += st[i].y * __builtin_amdgcn_exp2f(st[i].x - m);
    }
    for (int o = 1; o < P; o <<= 1) {
      const float m2 = __shfl_xor(m, o, 64), l2 = __shfl_xor(l, o, 64);
      const float mm = fmaxf(m, m2);
      float ls = 0.f;
      if (m > -INFINITY) ls += l * __builtin_amdgcn_exp2f(m - mm);
      if (m2 > -INFINITY) ls += l2 * __builtin_amdgcn_exp2f(m2 - mm);
      m = mm;
      l = ls;
    }
    if (hv && j == 0) {
      sM[h] = m;
      sL[h] = l;
    }
  }
  __syncthreads();
  // key-norm scores: this step's token adds -|k_new| / W (norm over all KV heads)
  // to its window, found by the block holding that window's list position
  int kn_pos = -1;
  float kn_delta = 0.f;
  if (MS == kScoreKeyNorm && a.T - 1 >= G.sink) {
    kn_pos = n_fq + ((a.T - 1 - G.sink) / G.W - a.ring_w0);
    if (blk - nh == kn_pos / per_blk) {   // uniform per block
      const uint16_t* kn = a.k_new + (int64_t)b * G.H_kv * kHeadDim;
      float sq = 0.f;
      for (int i = tid; i < G.H_kv * kHeadDim; i += kMergeThreads) {
        const float x = bf16_to_f32(kn[i]);
        sq = fmaf(x, x, sq);
      }
      skn[tid] = sq;
      __syncthreads();
      for (int o = kMergeThreads / 2; o > 0; o >>= 1) {
        if (tid < o) skn[tid] += skn[tid + o];
        __syncthreads();
      }
      kn_delta = -sqrtf(skn[0]) / (float)G.W;
    }
  }
  const int n_all = n_fq + a.n_ring + a.n_sink_items;
  const bool active = in_blk && pos < n_all;
  const float mass = (active && sL[hh] > 0.f && mr.x > -INFINITY)
                         ? __builtin_amdgcn_exp2f(mr.x - sM[hh]) * mr.y / sL[hh] : 0.f;
  // sum over the heads of the item: adjacent heads first (the heads of one KV
  // group), then the groups; a butterfly when H_q is a power of two
  float tot = mass;
  const bool pow2 = (nh & (nh - 1)) == 0;
  if (pow2) {
    for (int o = 1; o < nh; o <<= 1) tot += __shfl_xor(tot, o, 64);
  } else {
    smass[tid] = mass;
    __syncthreads();
    if (hh == 0 && in_blk) {
      const float* m = smass + li * nh;
      tot = 0.f;
      for (int g = 0; g < G.H_kv; ++g) {
        float sg = 0.f;
        for (int j = 0; j < G.gqa; ++j) sg += m[g * G.gqa + j];
        tot += sg;
      }
    }
  }
  if (!active) return;
  const int win = pos < n_fq ? wl : (pos < n_fq + a.n_ring ? a.ring_w0 + (pos - n_fq) : -1);
  if (G.flags & 2u) {   // per-head masses of this step, for inspection
    float* dbg = (float*)(ub + a.L.dbg_mass);
    const int w_h = pos < n_fq ? iwin[pos] : win;
    if (w_h >= 0) dbg[(int64_t)hh * (G.nwc + 1) + w_h] = mass;
    else atomicAdd(&dbg[(int64_t)hh * (G.nwc + 1) + G.nwc], mass);
  }
  if (hh == 0 && win >= 0) {
    float ns;
    if constexpr (MS == kScoreKeyNorm) {
      ns = old_score + (pos == kn_pos ? kn_delta : 0.f);
    } else if constexpr (MS == kScorePNorm) {
      // p-norm: {sum of completed periods' u^p, u of this period}; the score
      // is their sum with u^p.  A period's first step closes the previous one,
      // whose u^p the old score already includes.
      float2* pu = (float2*)(ub + a.L.pnorm) + win;
      float2 st = a.period_start ? make_float2(old_score, 0.f) : *pu;
      st.y += tot / (float)nh;
      ns = st.x + powf(st.y, a.pnorm_p);
      *pu = st;
    } else {
      ns = old_score * a.decay + tot / (float)nh;
    }
    ((float*)(ub + a.L.score))[win] = ns;
    iscore[pos] = ns;   // the next re-rank and merge read it by list position
  }
}

}  // namespace qv

// ---- launchers -------------------------------------------------------------
namespace qv {
template <int W, int NHS, bool ROPE>
hipError_t launch_attend_t(const AttnArgs& a, hipStream_t st) {
  dim3 grid(a.g.n_split, a.g.H_kv, a.g.B);
  const size_t smem = attn_smem_fixed<W, NHS, ROPE>() + 4 * (size_t)(a.g.max_fq + 1);
  if (smem > 160 * 1024) return hipErrorInvalidValue;   // live list too long for the LDS
  hipLaunchKernelGGL((k_attend<W, NHS, 2, ROPE>), grid, dim3(kAttnThreads), smem, st, a);
  return hipGetLastError();
}

// Calls f(W, NHS, ROPE) (integral constants) for the attention instantiation of a
// geometry: window size, 16-row head sets per KV head, RoPE-aware quantized tier.
template <class F>
hipError_t attend_variant(const Geometry& g, F&& f) {
  const int nhs = (g.gqa + 3) / 4;
  auto by_heads = [&](auto w, auto rope) -> hipError_t {
    if (nhs == 1) return f(w, std::integral_constant<int, 1>{}, rope);
    if (nhs == 2) return f(w, std::integral_constant<int, 2>{}, rope);
    return f(w, std::integral_constant<int, 4>{}, rope);
  };
  using T = std::true_type;
  using Fa = std::false_type;
  if (g.rope) {
    if (g.W == 32) return by_heads(std::integral_constant<int, 32>{}, T{});
    return by_heads(std::integral_constant<int, 64>{}, T{});
  }
  if (g.W == 8) return by_heads(std::integral_constant<int, 8>{}, Fa{});
  if (g.W == 32) return by_heads(std::integral_constant<int, 32>{}, Fa{});
  return by_heads(std::integral_constant<int, 64>{}, Fa{});
}

hipError_t launch_attend(const AttnArgs& a, hipStream_t st) {
  return attend_variant(a.g, [&](auto w, auto nhs, auto rope) {
    return launch_attend_t<decltype(w)::value, decltype(nhs)::value, decltype(rope)::value>(a, st);
  });
}

// Registers per lane and LDS bytes per workgroup of the attention kernel a
// geometry launches.
hipError_t attend_footprint(const Geometry& g, int* vgprs, size_t* lds) {
  return attend_variant(g, [&](auto w, auto nhs, auto rope) {
    constexpr int Wv = decltype(w)::value, Nv = decltype(nhs)::value;
    constexpr bool Rv = decltype(rope)::value;
    hipFuncAttributes fa;
    hipError_t e = hipFuncGetAttributes(&fa, reinterpret_cast<const void*>(&k_attend<Wv, Nv, 2, Rv>));
    if (e != hipSuccess) return e;
    *vgprs = fa.numRegs;
    *lds = fa.sharedSizeBytes + attn_smem_fixed<Wv, Nv, Rv>() + 4 * (size_t)(g.max_fq + 1);
    return hipSuccess;
  });
}

hipError_t launch_merge(const AttnArgs& a, hipStream_t st) {
  const int per_blk = kMergeThreads / a.g.H_q;
  const int n_mass = (a.g.max_items + per_blk - 1) / per_blk;
  dim3 grid(a.g.H_q + n_mass, a.g.B);
  const int need = (a.g.n_split + kSplitGroups - 1) / kSplitGroups;
  auto go = [&](auto kern) { hipLaunchKernelGGL(kern, grid, dim3(kMergeThreads), 0, st, a); };
  auto by_split = [&](auto ms) {
    constexpr int MS = decltype(ms)::value;
    if (need <= 4) go(k_merge<4, MS>);
    else if (need <= 8) go(k_merge<8, MS>);
    else go(k_merge<32, MS>);
  };
  if (a.key_norm) by_split(std::integral_constant<int, kScoreKeyNorm>{});
  else if (a.pnorm_p > 0.f) by_split(std::integral_constant<int, kScorePNorm>{});
  else by_split(std::integral_constant<int, kScoreMass>{});
  return hipGetLastError();
}
}  // namespace qv
