// Window migrations between the tier pools (QEvict Sec. 4.3, migration-stable
// quantization; Algorithm 1 promote / quantize-once steps), driven by the work
// lists the re-tier kernel wrote; grids are sized for the worst case and idle
// workgroups exit at once, so no host synchronisation is needed.
//
// Quantization of one group x (asymmetric, b bits, n = 2^b - 1 levels):
//   z = largest fp16 <= min(x); s = smallest fp16 >= 0 with z + n s >= max(x);
//   c = round-half-even((x - z) / s)   (all codes 0 when s = 0).
// z + k s / 2 is exact in float64 for the integers k involved (fp16 operands),
// so every comparison that decides s or a code is exact and the result is
// bit-identical to the definition.  Keys form one group per channel across the
// window's tokens, values one group per token across G channels.
// Promotion writes RNE_bf16(z + s c), with z + s c formed exactly in float64.
#include "qv_device.h"

namespace qv {

__device__ __forceinline__ bool quant_params(float lo, float hi, int nbits, uint16_t* zb, uint16_t* sb) {
  if (!(lo >= -65504.f && hi <= 65504.f)) return false;   // also rejects NaN
  const uint16_t zh = fp16_round_down(lo);
  const double z = fp16_bits_to_f64(zh);
  const double n = (double)((1 << nbits) - 1);
  const double hid = hi;
  const float t = (float)((hid - z) / n);
  uint16_t sh = __builtin_bit_cast(uint16_t, (_Float16)t);
  for (int k = 0; k < 8 && z + fp16_bits_to_f64(sh) * n < hid; ++k) sh = fp16_next_up(sh);
  for (int k = 0; k < 8 && sh != 0 && z + fp16_bits_to_f64(fp16_next_down(sh)) * n >= hid; ++k)
    sh = fp16_next_down(sh);
  *zb = zh;
  *sb = sh;
  return true;
}

// Parameters of one quantization group as the code pass uses them: fp16 zero
// and scale widened to fp32 (exact) and the fp32 reciprocal of the scale.
struct QParams {
  float z, s, inv_s, pad;
};

__device__ __forceinline__ QParams group_params(float lo, float hi, int nbits, uint16_t* zb, uint16_t* sb,
                                int32_t* counts) {
  if (!quant_params(lo, hi, nbits, zb, sb)) set_error(counts, ERR_RANGE);
  QParams p;
  const double z = fp16_bits_to_f64(*zb), s = fp16_bits_to_f64(*sb);
  p.z = (float)z;
  p.s = (float)s;
  p.inv_s = s > 0.0 ? 1.f / (float)s : 0.f;
  p.pad = 0.f;
  return p;
}

// Round-half-even code of x in the group: an fp32 estimate of (x - z) / s
// (within one of the exact result), then the exact decision against the
// neighbouring half-step boundaries z + (c +- 1/2) s, formed in float64 where
// they are exact (fp16 operands, |c| <= 16).  Written without branches or
// selects between paths, so that the codes of a lane's entries and their
// parameter loads overlap.
__device__ __forceinline__ uint32_t quant_code(float x, const QParams& p, int nmax) {
  const float nm = (float)nmax;
  float c = rintf((x - p.z) * p.inv_s);
  c = fminf(fmaxf(c, 0.f), nm);
  const int odd = ((int)c) & 1;
  const double xd = x, cd = c, zd = p.z, sd = p.s;
  const double hi = zd + (cd + 0.5) * sd, lo = zd + (cd - 0.5) * sd;
  const int up = ((xd > hi) | ((xd == hi) & odd)) & (c < nm);
  const int dn = ((xd < lo) | ((xd == lo) & odd)) & (c > 0.f);
  c += (float)(up - dn);   // at most one of the two holds
  return p.s == 0.f ? 0u : (uint32_t)c;
}

// A (window, KV head) migration is split into four parts, one per workgroup
// pass: part = 2 area + h, area 0 the keys and 1 the values, h the channel half
// [64 h, 64 h + 64).  Key groups (one channel), value groups (one token, G
// channels, G = W), bf16 chunks and code words each fall in exactly one part:
// key entry / chunk e has channel block 32 (e & 3), value entry / chunk e has
// channel block 16 (e & 7), and an int2 word's two entries share their half.
constexpr int kParts = 4;
// value group (channels) of a window length: G = W, except 32 for 8-token windows
template <int W>
constexpr int value_group() { return W == 8 ? 32 : W; }
// LDS row of one token's 128 channels, padded by 16 bytes so that 16-byte
// accesses to 16 consecutive tokens fall in distinct banks
constexpr int kLdsRow = kHeadDim + 8;
// bf16 chunk (= code entry) index of local chunk cl of channel half h of an area
__device__ __forceinline__ int part_chunk(int area, int h, int cl) {
  return area == 0 ? (cl >> 1) * 4 + 2 * h + (cl & 1) : (cl >> 2) * 8 + 4 * h + (cl & 3);
}
// With RoPE a pre-RoPE key channel depends on both channel halves, so the key
// work of a window is not split: part 0 takes both halves, part 1 none.  The
// channel halves a part covers: [h0, h0 + nh).
struct Halves {
  int h0, nh;
};
template <bool ROPE>
__device__ __forceinline__ Halves part_halves(int area, int h) {
  if (ROPE && area == 0) return Halves{0, h == 0 ? 2 : 0};
  return Halves{h, 1};
}
// RoPE (cos, sin) of position p, channel pair i
__device__ __forceinline__ float2 rope_cs(const Geometry& G, int p, int i) {
  return *(const float2*)(G.rope + 2 * ((int64_t)p * (kHeadDim / 2) + i));
}

// Codes of one (window, KV head), packed: thread (area, block m, lane L, word
// comp) forms word 4m + comp of lane L; entry e of a word holds its 8 codes at
// bits 16 o + NB (4 e' + i) for code j = 2i + o.  Consecutive threads write
// consecutive words.
// 256 threads and, for 32-token windows, at most 96 VGPRs (five waves per SIMD):
// a migration workgroup fits on a compute unit beside two attention workgroups,
// so routing on its own stream does not hold back the attention of the next layers
constexpr int kMigrateThreads = 256;
// (the RoPE variants hold both key halves and their rotation: one wave fewer)
template <int W, bool ROPE = false>
constexpr int migrate_waves_per_simd() { return (W <= 32 ? 5 : 4) - (ROPE ? 1 : 0); }

template <int W, int NB, bool ROPE>
__device__ __forceinline__ void pack_codes(const Geometry& G, const uint16_t* sk, const uint16_t* sv,
                                           const QParams* pk, const QParams* pv, uint8_t* rec, int tid,
                                           int part) {
  constexpr int NBLK = W * NB / 64;
  constexpr int PER = 4 / NB;
  constexpr int NG = kHeadDim / W;
  constexpr int nmax = (1 << NB) - 1;
  const int area = part >> 1, h = part & 1;
  // Only the words this part owns are enumerated, one word (m, comp) per wave
  // pass, so that every lane of a wave forms codes (entry halves: keys by
  // (e & 3) >> 1, values by (e & 7) >> 2; with RoPE part 0 takes every key word)
  const bool all_keys = ROPE && area == 0;
  const int n_own = all_keys ? (h == 0 ? NBLK * 4 : 0) : NBLK * 2;
  for (int u = tid; u < n_own * 64; u += kMigrateThreads) {
    const int L = u & 63, o = u >> 6;
    int m, comp;
    if (all_keys) {
      m = o >> 2;
      comp = o & 3;
    } else if (area == 0) {
      m = o >> 1;
      comp = NB == 4 ? 2 * h + (o & 1) : h + 2 * (o & 1);
    } else if (NB == 4) {
      m = 2 * (o >> 2) + h;
      comp = o & 3;
    } else {
      m = o >> 1;
      comp = 2 * h + (o & 1);
    }
    const int q = L >> 4, r = L & 15;
    uint32_t wd = 0;
#pragma unroll
    for (int ee = 0; ee < PER; ++ee) {
      const int ei = (m * 4 + comp) * PER + ee;
      if (area == 0) {   // key entry (tb, kb): token 16 tb + r, channels 32 kb + 8 q + j
        const int t = 16 * (ei >> 2) + r, c0 = 32 * (ei & 3) + 8 * q;
        const u32x4 v = *(const u32x4*)(sk + t * kLdsRow + c0);
        const uint32_t vw[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float x = bf16_to_f32((uint16_t)(vw[j >> 1] >> (16 * (j & 1))));
          wd |= quant_code(x, pk[c0 + j], nmax) << ((j & 1) * 16 + NB * (4 * ee + (j >> 1)));
        }
      } else {           // value entry (kt, cb): token tok(kt, q, j), channel 16 cb + r
        const int kt = ei >> 3, c = 16 * (ei & 7) + r, vg = c / W;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int t = v_tok(kt, q, j);
          const float x = bf16_to_f32(sv[t * kLdsRow + c]);
          wd |= quant_code(x, pv[t * NG + vg], nmax) << ((j & 1) * 16 + NB * (4 * ee + (j >> 1)));
        }
      }
    }
    *(uint32_t*)(rec + area * G.qcodes_bytes + ((int64_t)m * 64 + L) * 16 + comp * 4) = wd;
  }
}

// Codes of one KV head of an 8-token window (layout of the header): thread
// (lane, word) of this part forms one 32-bit word.  Keys: lane (q, r < 8) of
// token r, words of channel blocks kb = 2 h, 2 h + 1 (int2: one word holding
// both); values: lane (q < 2, r), words of channel-block pairs cp = 2 h, 2 h + 1
// (int2: one word), value group cp.
template <int NB>
__device__ __forceinline__ void pack_codes8(const Geometry& G, const uint16_t* sk, const uint16_t* sv,
                                            const QParams* pk, const QParams* pv, uint8_t* rec, int tid,
                                            int part) {
  constexpr int nmax = (1 << NB) - 1;
  constexpr int WPH = NB == 4 ? 2 : 1;    // words of a lane in one channel half
  constexpr int LB = NB == 4 ? 16 : 8;    // code bytes of a lane
  constexpr int NG = kHeadDim / 32;
  const int area = part >> 1, h = part & 1;
  if (tid >= 32 * WPH) return;
  const int ln = tid % 32, wl = tid / 32;
  const int word = WPH * h + wl;          // int4: block kb / pair cp; int2: the half's word
  uint32_t wd = 0;
  if (area == 0) {
    const int q = ln >> 3, r = ln & 7;    // token r, channels 32 kb + 8 q + j
#pragma unroll
    for (int ee = 0; ee < 4 / NB; ++ee) {
      const int kb = NB == 4 ? word : 2 * word + ee;
      const int c0 = 32 * kb + 8 * q;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float x = bf16_to_f32(sk[r * kLdsRow + c0 + j]);
        wd |= quant_code(x, pk[c0 + j], nmax) << ((j & 1) * 16 + NB * (4 * ee + (j >> 1)));
      }
    }
    *(uint32_t*)(rec + (q * 8 + r) * LB + 4 * word) = wd;
  } else {
    const int q = ln >> 4, r = ln & 15;   // tokens 4 q + j, channel 16 cb + r
#pragma unroll
    for (int ee = 0; ee < 4 / NB; ++ee) {
      const int cp = NB == 4 ? word : 2 * word + ee;
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int t = 4 * q + j, c = 16 * (2 * cp + e) + r;
          const float x = bf16_to_f32(sv[t * kLdsRow + c]);
          wd |= quant_code(x, pv[t * NG + cp], nmax) << ((j & 1) * 16 + NB * (4 * ee + 2 * e + (j >> 1)));
        }
    }
    *(uint32_t*)(rec + G.qcodes_bytes + (q * 16 + r) * LB + 4 * word) = wd;
  }
}

// Load one part of one KV head of a window into LDS in natural [t][c] layout.
template <int W, bool ROPE>
__device__ __forceinline__ void load_window(const MigrateArgs& a, uint8_t* ub, int b, int g, int w, int src_kind,
                            int src_idx, uint16_t* sk, uint16_t* sv, int part) {
  const Geometry& G = a.g;
  const int tid = threadIdx.x;
  const int area = part >> 1, h = part & 1;
  const Halves hv = part_halves<ROPE>(area, h);
  uint16_t* dst = area == 0 ? sk : sv;
  if (src_kind == SRC_PROMPT) {
    const int64_t row0 = ((int64_t)b * G.H_kv + g) * a.src_T + G.sink + (int64_t)w * W;
    const uint16_t* src = (area == 0 ? a.src_k : a.src_v) + row0 * kHeadDim;
    for (int i = tid; i < W * 8 * hv.nh; i += blockDim.x) {
      const int t = (i >> 3) % W, c = 64 * (hv.h0 + i / (W * 8)) + 8 * (i & 7);
      *(u32x4*)(dst + t * kLdsRow + c) = *(const u32x4*)(src + t * kHeadDim + c);
    }
  } else if constexpr (W == 8) {
    // 16-byte pieces of this half: keys (kb, q, r < 8), values (cp, q < 2, r)
    const uint8_t* p = ub + (src_kind == SRC_FSLOT ? a.L.fpool : a.L.ring) +
                       (int64_t)src_idx * G.fslot_bytes + g * G.fhead_bytes;
    for (int i = tid; i < 64; i += blockDim.x) {
      if (area == 0) {
        const int kb = 2 * h + (i >> 5), q = (i >> 3) & 3, r = i & 7;
        *(u32x4*)(sk + r * kLdsRow + 32 * kb + 8 * q) = *(const u32x4*)(p + ((kb * 4 + q) * 8 + r) * 16);
      } else {
        const int cp = 2 * h + (i >> 5), q = (i >> 4) & 1, r = i & 15;
        const u32x4 x = *(const u32x4*)(p + (int64_t)W * kHeadDim * 2 + ((cp * 2 + q) * 16 + r) * 16);
        const uint32_t vw[4] = {x[0], x[1], x[2], x[3]};
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            sv[(4 * q + j) * kLdsRow + 16 * (2 * cp + e) + r] =
                (uint16_t)(vw[2 * e + (j >> 1)] >> (16 * (j & 1)));
      }
    }
  } else {
    const uint8_t* p = ub + (src_kind == SRC_FSLOT ? a.L.fpool : a.L.ring) +
                       (int64_t)src_idx * G.fslot_bytes + g * G.fhead_bytes +
                       (area == 0 ? 0 : (int64_t)W * kHeadDim * 2);
    // K chunk (tb, kb), lane 16q + r: token 16 tb + r, channels 32 kb + 8 q .. + 7
    // V chunk (kt, cb), lane 16q + r: tokens tok(kt, q, 0..7), channel 16 cb + r
    for (int i = tid; i < (W / 8) * 64 * hv.nh; i += blockDim.x) {
      const int ih = i / ((W / 8) * 64), il = i % ((W / 8) * 64);
      const int chunk = part_chunk(area, hv.h0 + ih, il >> 6), L = il & 63, q = L >> 4, r = L & 15;
      const u32x4 x = *(const u32x4*)(p + ((int64_t)chunk * 64 + L) * 16);
      if (area == 0) {
        *(u32x4*)(sk + (16 * (chunk >> 2) + r) * kLdsRow + 32 * (chunk & 3) + 8 * q) = x;
      } else {
        const int kt = chunk >> 3, c = 16 * (chunk & 7) + r;
        const uint32_t vw[4] = {x[0], x[1], x[2], x[3]};
#pragma unroll
        for (int j = 0; j < 8; ++j)
          sv[v_tok(kt, q, j) * kLdsRow + c] = (uint16_t)(vw[j >> 1] >> (16 * (j & 1)));
      }
    }
  }
}

// One (window, KV head) task per workgroup pass: (1) the window into LDS,
// (2) one thread per group: min / max, scale and zero (written to the record),
// (3) one thread per (code block, lane): the codes of its entries straight into
// the packed 16-byte block (entry e's 8 codes at bits 16 o + b (4 e' + i)).
// Keys form groups per channel (W tokens), values per token (G = W channels).
// One work-list entry (win, src_kind, src_idx, dst, bits, dep), held in registers.
struct WorkEntry {
  int32_t v[kQEntry];
};
__device__ __forceinline__ WorkEntry load_entry(const int32_t* list, int e) {
  WorkEntry x;
#pragma unroll
  for (int i = 0; i < kQEntry; ++i) x.v[i] = list[e * kQEntry + i];
  return x;
}

// Pre-RoPE keys of a window held in LDS ([t][c] bf16, both halves, absolute
// position of token t = p0 + t): channel i < 64 becomes x_i cos + x_{i+64} sin,
// channel i + 64 becomes x_{i+64} cos - x_i sin, each product and sum rounded to
// float32 (no fused multiply-add), then RNE to bf16.  All values are read
// before any is written.
template <int W>
__device__ __forceinline__ void unrotate_keys(const Geometry& G, uint16_t* sk, int p0, int tid) {
#pragma clang fp contract(off)
  constexpr int PER = W * 64 / kMigrateThreads;   // channel pairs per thread
  uint16_t lo[PER], hi[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = tid + k * kMigrateThreads, t = e / 64, i = e % 64;
    const float a = bf16_to_f32(sk[t * kLdsRow + i]), bb = bf16_to_f32(sk[t * kLdsRow + 64 + i]);
    const float2 cs = rope_cs(G, p0 + t, i);
    const float ac = a * cs.x, bs = bb * cs.y, bc = bb * cs.x, as = a * cs.y;
    lo[k] = f32_to_bf16_rne(ac + bs);
    hi[k] = f32_to_bf16_rne(bc - as);
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = tid + k * kMigrateThreads, t = e / 64, i = e % 64;
    sk[t * kLdsRow + i] = lo[k];
    sk[t * kLdsRow + 64 + i] = hi[k];
  }
}

template <int W>
struct QuantLds {
  uint16_t sk[W * kLdsRow];
  uint16_t sv[W * kLdsRow];
  QParams pk[kHeadDim];
  QParams pv[W * (kHeadDim / value_group<W>())];
};

template <int W, bool ROPE>
__device__ __forceinline__ void quantize_task(const MigrateArgs& a, uint8_t* ub, int b, int g,
                                              const WorkEntry& ent, QuantLds<W>& sm, int32_t* counts,
                                              int part) {
  const Geometry& G = a.g;
  constexpr int GV = value_group<W>();         // channels of a value group
  constexpr int NG = kHeadDim / GV;            // value groups per token
  constexpr int NGH = 64 / GV;                 // value groups per token in one channel half
  constexpr int NX = W > GV ? W : GV;          // values of the largest group
  const int tid = threadIdx.x;
  const int area = part >> 1, h = part & 1;
  const int w = ent.v[0], src_kind = ent.v[1], src_idx = ent.v[2], dst = ent.v[3], nb = ent.v[4];
  uint16_t* sk = sm.sk;
  uint16_t* sv = sm.sv;
  load_window<W, ROPE>(a, ub, b, g, w, src_kind, src_idx, sk, sv, part);
  __syncthreads();
  const Halves hv = part_halves<ROPE>(area, h);
  if (ROPE && area == 0 && hv.nh == 2) {
    unrotate_keys<W>(G, sk, G.sink + w * W, tid);
    __syncthreads();
  }
  uint8_t* rec = ub + a.L.qpool + (int64_t)dst * G.qslot_bytes + g * G.qrec_bytes;
  // ---- group parameters: one thread per group of this part (keys: 64 channels
  // per half; values: W tokens x NGH groups per half) ----
  const int n_groups = area == 0 ? 64 * hv.nh : W * NGH;
  if (tid < n_groups) {
    float x[NX];
    int c = 0, t = 0, vg = 0;
    const int n = area == 0 ? W : GV;   // values in the group
    if (area == 0) {
      c = 64 * hv.h0 + tid;
#pragma unroll
      for (int tt = 0; tt < W; ++tt) x[tt] = bf16_to_f32(sk[tt * kLdsRow + c]);
    } else {
      t = tid / NGH;
      vg = NGH * h + tid % NGH;
      const u32x4* row = (const u32x4*)(sv + t * kLdsRow + vg * GV);
#pragma unroll
      for (int k = 0; k < GV / 8; ++k) {
        const u32x4 v = row[k];
        const uint32_t vw[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
        for (int i = 0; i < 8; ++i) x[8 * k + i] = bf16_to_f32((uint16_t)(vw[i >> 1] >> (16 * (i & 1))));
      }
    }
    float lo = x[0], hi = x[0];
#pragma unroll
    for (int i = 1; i < NX; ++i) {
      if (i < n) {
        lo = fminf(lo, x[i]);
        hi = fmaxf(hi, x[i]);
      }
    }
    uint16_t zb = 0, sb = 0;
    const QParams p = group_params(lo, hi, nb, &zb, &sb, counts);
    if (area == 0) {
      sm.pk[c] = p;
      uint16_t* mk = (uint16_t*)(rec + meta_k_off(G));
      mk[c] = sb;
      mk[kHeadDim + c] = zb;
    } else {
      sm.pv[t * NG + vg] = p;
      uint8_t* mv = rec + meta_v_elem(G, t, vg);
      *(uint16_t*)mv = sb;
      *(uint16_t*)(mv + meta_v_zero_delta(G)) = zb;
    }
  }
  __syncthreads();
  // ---- codes, packed ----
  if constexpr (W == 8) {
    if (nb == 4) pack_codes8<4>(G, sk, sv, sm.pk, sm.pv, rec, tid, part);
    else pack_codes8<2>(G, sk, sv, sm.pk, sm.pv, rec, tid, part);
  } else {
    if (nb == 4) pack_codes<W, 4, ROPE>(G, sk, sv, sm.pk, sm.pv, rec, tid, part);
    else pack_codes<W, 2, ROPE>(G, sk, sv, sm.pk, sm.pv, rec, tid, part);
  }
}

// 8 bf16 values z_j + s_j c_j (exact in float64, one rounding) packed for a 16-byte store
template <int NB>
__device__ __forceinline__ u32x4 dequant8(uint32_t wd, int ee, u32x4 s8, u32x4 z8) {
  constexpr uint32_t mask = (1u << NB) - 1u;
  const uint32_t sw[4] = {s8[0], s8[1], s8[2], s8[3]};
  const uint32_t zw[4] = {z8[0], z8[1], z8[2], z8[3]};
  uint32_t outw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t pair = 0;
#pragma unroll
    for (int o = 0; o < 2; ++o) {
      const uint32_t code = (wd >> (o * 16 + NB * (4 * ee + i))) & mask;
      const double sj = fp16_bits_to_f64((uint16_t)(sw[i] >> (16 * o)));
      const double zj = fp16_bits_to_f64((uint16_t)(zw[i] >> (16 * o)));
      pair |= (uint32_t)f64_to_bf16_rne(zj + sj * (double)code) << (16 * o);
    }
    outw[i] = pair;
  }
  return (u32x4){outw[0], outw[1], outw[2], outw[3]};
}

// z + s c (exact in float64) of key entry e (channels 32 (e & 3) + 8 q .. + 7 of
// token 16 (e >> 2) + r) for lane L = 16 q + r
template <int NB>
__device__ __forceinline__ void key_entry_f64(const Geometry& G, const uint8_t* rec, int e, int L,
                                              double (&x)[8]) {
  constexpr int PER = 4 / NB;
  constexpr uint32_t mask = (1u << NB) - 1u;
  const int q = L >> 4, word = e / PER, ee = e % PER;
  const uint32_t wd = *(const uint32_t*)(rec + ((int64_t)(word >> 2) * 64 + L) * 16 + (word & 3) * 4);
  const uint8_t* ps = rec + meta_k_off(G) + 2 * (32 * (e & 3) + 8 * q);
  const u32x4 s8 = *(const u32x4*)ps, z8 = *(const u32x4*)(ps + 2 * kHeadDim);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int o = 0; o < 2; ++o) {
      const uint32_t code = (wd >> (o * 16 + NB * (4 * ee + i))) & mask;
      const double sj = fp16_bits_to_f64((uint16_t)(s8[i] >> (16 * o)));
      const double zj = fp16_bits_to_f64((uint16_t)(z8[i] >> (16 * o)));
      x[2 * i + o] = zj + sj * (double)code;
    }
}

// Promoted bf16 keys of entry e with RoPE: the dequantized pre-RoPE keys of the
// entry and of its partner entry e ^ 2 (channels +- 64) rotated to position
// p0 + token: channel i < 64 takes x_i cos - x_{i+64} sin, channel i + 64 takes
// x_{i+64} cos + x_i sin, products and sums rounded in float64, then RNE to bf16.
template <int NB>
__device__ __forceinline__ u32x4 rope_key8(const Geometry& G, const uint8_t* rec, int e, int L, int p0) {
#pragma clang fp contract(off)
  double x[8], y[8];
  key_entry_f64<NB>(G, rec, e, L, x);
  key_entry_f64<NB>(G, rec, e ^ 2, L, y);
  const int kb = e & 3, q = L >> 4, r = L & 15;
  const int p = p0 + 16 * (e >> 2) + r;
  uint32_t outw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t pair = 0;
#pragma unroll
    for (int o = 0; o < 2; ++o) {
      const int j = 2 * i + o;
      const float2 cs = rope_cs(G, p, (32 * kb + 8 * q + j) & 63);
      const double t1 = x[j] * (double)cs.x, t2 = y[j] * (double)cs.y;
      const double v = kb < 2 ? t1 - t2 : t1 + t2;
      pair |= (uint32_t)f64_to_bf16_rne(v) << (16 * o);
    }
    outw[i] = pair;
  }
  return (u32x4){outw[0], outw[1], outw[2], outw[3]};
}

// Promotion of one (window, KV head) from its quantized record: thread (area,
// entry e, lane L) loads the 32-bit code word holding entry e of lane L and the
// entry's 8 scales and zeros, and writes its 8 bf16 values to the same
// (entry, lane) position of the bf16 slot.
template <int W, int NB, bool ROPE>
__device__ __forceinline__ void promote_from_record(const Geometry& G, const uint8_t* rec,
                                                    uint8_t* dp, int tid, int part, int p0) {
  constexpr int E = W / 4;                          // entries per area
  constexpr int PER = 4 / NB;
  const int ng = kHeadDim / G.G;
  const int area = part >> 1, h = part & 1;
  // only the entries this part owns, one per wave pass (see pack_codes)
  const bool all_keys = ROPE && area == 0;
  const int n_own = all_keys ? (h == 0 ? E : 0) : E / 2;
  for (int tk = tid; tk < n_own * 64; tk += kMigrateThreads) {
    const int L = tk & 63, o = tk >> 6;
    const int ei = all_keys ? o : (area == 0 ? 4 * (o >> 1) + 2 * h + (o & 1) : 8 * (o >> 2) + 4 * h + (o & 3));
    if (ROPE && area == 0) {
      *(u32x4*)(dp + ((int64_t)ei * 64 + L) * 16) = rope_key8<NB>(G, rec, ei, L, p0);
      continue;
    }
    const int q = L >> 4, r = L & 15;
    const int word = ei / PER;
    const uint32_t wd = *(const uint32_t*)(rec + area * G.qcodes_bytes +
                                           ((int64_t)(word >> 2) * 64 + L) * 16 + (word & 3) * 4);
    const uint8_t* ps;
    u32x4 s8, z8;
    if (area == 0) {   // key entry (tb, kb): channels 32 kb + 8 q .. + 7
      ps = rec + meta_k_off(G) + 2 * (32 * (ei & 3) + 8 * q);
      s8 = *(const u32x4*)ps;
      z8 = *(const u32x4*)(ps + 2 * kHeadDim);
    } else {           // value entry (kt, cb): tokens tok(kt, q, 0..7), channel 16 cb + r
      const int c = 16 * (ei & 7) + r;
      ps = rec + meta_v_off(G) + (((ei >> 3) * 4 + q) * ng + c / G.G) * 32;
      s8 = *(const u32x4*)ps;
      z8 = *(const u32x4*)(ps + 16);
    }
    const int64_t off = (area == 0 ? 0 : (int64_t)W * kHeadDim * 2) + ((int64_t)ei * 64 + L) * 16;
    *(u32x4*)(dp + off) = dequant8<NB>(wd, ei % PER, s8, z8);
  }
}

// Promotion of one KV head of an 8-token window from its record: one thread per
// 16-byte piece of this part's half (keys: block kb, lane (q, r < 8); values:
// block pair cp, lane (q < 2, r)), its values z + s c formed exactly in float64
// and rounded once to bf16.
template <int NB>
__device__ __forceinline__ void promote_from_record8(const Geometry& G, const uint8_t* rec, uint8_t* dp,
                                                     int tid, int part) {
  constexpr uint32_t mask = (1u << NB) - 1u;
  constexpr int LB = NB == 4 ? 16 : 8;
  const int area = part >> 1, h = part & 1;
  if (tid >= 64) return;
  uint32_t outw[4];
  if (area == 0) {
    const int kb = 2 * h + (tid >> 5), q = (tid >> 3) & 3, r = tid & 7;
    const int word = NB == 4 ? kb : kb >> 1, ee = NB == 4 ? 0 : kb & 1;
    const uint32_t wd = *(const uint32_t*)(rec + (q * 8 + r) * LB + 4 * word);
    const uint8_t* ps = rec + meta_k_off(G) + 2 * (32 * kb + 8 * q);
    const u32x4 s8 = *(const u32x4*)ps, z8 = *(const u32x4*)(ps + 2 * kHeadDim);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t pair = 0;
#pragma unroll
      for (int o = 0; o < 2; ++o) {
        const uint32_t code = (wd >> (o * 16 + NB * (4 * ee + i))) & mask;
        const double sj = fp16_bits_to_f64((uint16_t)(s8[i] >> (16 * o)));
        const double zj = fp16_bits_to_f64((uint16_t)(z8[i] >> (16 * o)));
        pair |= (uint32_t)f64_to_bf16_rne(zj + sj * (double)code) << (16 * o);
      }
      outw[i] = pair;
    }
    *(u32x4*)(dp + ((kb * 4 + q) * 8 + r) * 16) = (u32x4){outw[0], outw[1], outw[2], outw[3]};
  } else {
    const int cp = 2 * h + (tid >> 5), q = (tid >> 4) & 1, r = tid & 15;
    const int word = NB == 4 ? cp : cp >> 1, ee = NB == 4 ? 0 : cp & 1;
    const uint32_t wd = *(const uint32_t*)(rec + G.qcodes_bytes + (q * 16 + r) * LB + 4 * word);
    // value group cp: scales then zero points of tokens 4 q .. 4 q + 3
    const u32x4 m = *(const u32x4*)(rec + meta_v_off(G) + (q * 4 + cp) * 16);
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int jp = 0; jp < 2; ++jp) {
        uint32_t pair = 0;
#pragma unroll
        for (int o = 0; o < 2; ++o) {
          const int j = 2 * jp + o;
          const uint32_t code = (wd >> (o * 16 + NB * (4 * ee + 2 * e + jp))) & mask;
          const double sj = fp16_bits_to_f64((uint16_t)(m[j >> 1] >> (16 * (j & 1))));
          const double zj = fp16_bits_to_f64((uint16_t)(m[2 + (j >> 1)] >> (16 * (j & 1))));
          pair |= (uint32_t)f64_to_bf16_rne(zj + sj * (double)code) << (16 * o);
        }
        outw[2 * e + jp] = pair;
      }
    *(u32x4*)(dp + (int64_t)8 * kHeadDim * 2 + ((cp * 2 + q) * 16 + r) * 16) =
        (u32x4){outw[0], outw[1], outw[2], outw[3]};
  }
}

template <int W, bool ROPE>
__device__ __forceinline__ void promote_task(const MigrateArgs& a, uint8_t* ub, int b, int g,
                                             const WorkEntry& ent, int part) {
  const Geometry& G = a.g;
  const int tid = threadIdx.x;
  const int area = part >> 1, h = part & 1;
  const int w = ent.v[0], src_kind = ent.v[1], src_idx = ent.v[2], dst = ent.v[3], nb = ent.v[4];
  uint8_t* dp = ub + a.L.fpool + (int64_t)dst * G.fslot_bytes + g * G.fhead_bytes;
  const int64_t area_off = area == 0 ? 0 : (int64_t)W * kHeadDim * 2;
  const Halves hv = part_halves<ROPE>(area, h);
  if (W == 8 && src_kind == SRC_RING) {
    // the half's 16-byte pieces: keys (kb, q, r < 8), values (cp, q < 2, r)
    const uint8_t* sp = ub + a.L.ring + (int64_t)src_idx * G.fslot_bytes + g * G.fhead_bytes;
    for (int i = tid; i < 64; i += blockDim.x) {
      const int64_t off = area == 0 ? (int64_t)(((2 * h + (i >> 5)) * 4 + ((i >> 3) & 3)) * 8 + (i & 7)) * 16
                                    : (int64_t)W * kHeadDim * 2 +
                                          (int64_t)(((2 * h + (i >> 5)) * 2 + ((i >> 4) & 1)) * 16 + (i & 15)) * 16;
      *(u32x4*)(dp + off) = *(const u32x4*)(sp + off);
    }
  } else if (src_kind == SRC_RING) {
    const uint8_t* sp = ub + a.L.ring + (int64_t)src_idx * G.fslot_bytes + g * G.fhead_bytes;
    for (int i = tid; i < (W / 8) * 64 * hv.nh; i += blockDim.x) {
      const int ih = i / ((W / 8) * 64), il = i % ((W / 8) * 64);
      const int64_t off = area_off + ((int64_t)part_chunk(area, hv.h0 + ih, il >> 6) * 64 + (il & 63)) * 16;
      *(u32x4*)(dp + off) = *(const u32x4*)(sp + off);
    }
  } else if (src_kind == SRC_PROMPT) {
    const int64_t row0 = ((int64_t)b * G.H_kv + g) * a.src_T + G.sink + (int64_t)w * W;
    if (area == 0) {
      const uint16_t* ks = a.src_k + row0 * kHeadDim;
      for (int i = tid; i < W * 8 * hv.nh; i += blockDim.x) {
        const int t = (i >> 3) % W, c = 64 * (hv.h0 + i / (W * 8)) + 8 * (i & 7);
        *(u32x4*)(dp + k_elem_off(W, t, c)) = *(const u32x4*)(ks + t * kHeadDim + c);
      }
    } else {
      const uint16_t* vs = a.src_v + row0 * kHeadDim;
      for (int i = tid; i < W * 64; i += blockDim.x) {
        const int t = i >> 6, c = 64 * h + (i & 63);
        *(uint16_t*)(dp + v_elem_off(W, t, c)) = vs[t * kHeadDim + c];
      }
    }
  } else {   // SRC_QSLOT
    const uint8_t* rec = ub + a.L.qpool + (int64_t)src_idx * G.qslot_bytes + g * G.qrec_bytes;
    const int p0 = G.sink + w * W;   // position of the window's first token
    if constexpr (W == 8) {
      if (nb == 4) promote_from_record8<4>(G, rec, dp, tid, part);
      else promote_from_record8<2>(G, rec, dp, tid, part);
    } else {
      if (nb == 4) promote_from_record<W, 4, ROPE>(G, rec, dp, tid, part, p0);
      else promote_from_record<W, 2, ROPE>(G, rec, dp, tid, part, p0);
    }
  }
}

// Migrations of one routing event, one (window, KV head, part) task per
// workgroup pass.  The first half of the grid takes the quantizations, the
// second half the promotions / admissions, so a workgroup knows its list before
// the counts arrive and reads the counts and its first entry in one round.  A
// promotion whose bf16 slot is being vacated by a quantization in the same event
// (dep >= 0) runs in that quantization's workgroup right after it, part by part,
// so the slot is read before it is overwritten without any ordering across
// workgroups.
template <int W, bool ROPE>
__global__ __launch_bounds__(kMigrateThreads, (migrate_waves_per_simd<W, ROPE>())) void k_migrate(MigrateArgs a) {
  const Geometry& G = a.g;
  const int b = blockIdx.y;
  __shared__ __attribute__((aligned(16))) QuantLds<W> sm;
  // a routing batch whose wait for the cache stream timed out moves nothing (the
  // word is read with the first loads)
  const int gate_failed =
      a.gate_fail ? __hip_atomic_load(a.gate_fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
  uint8_t* ub = a.base[blockIdx.z] + (int64_t)b * a.L.unit_bytes;
  int32_t* counts = (int32_t*)(ub + a.L.counts);
  const int32_t* qlist = (const int32_t*)(ub + a.L.qlist);
  const int32_t* plist = (const int32_t*)(ub + a.L.plist);
  const int half = gridDim.x / 2;
  const bool quant = (int)blockIdx.x < half;
  const int x0 = quant ? blockIdx.x : blockIdx.x - half;
  const int32_t* list = quant ? qlist : plist;
  const int per_entry = G.H_kv * kParts;
  const int e0 = x0 / per_entry;
  const WorkEntry first = load_entry(list, e0 <= G.max_fq ? e0 : 0);   // lists hold max_fq + 1 entries
  const int n_tasks = gate_failed ? 0 : (quant ? counts[CNT_QUANT] : counts[CNT_PROMOTE]) * per_entry;
  for (int task = x0; task < n_tasks; task += half) {
    const int e = task / per_entry, g = (task / kParts) % G.H_kv, part = task % kParts;
    const WorkEntry ent = task == x0 ? first : load_entry(list, e);
    if (quant) {
      quantize_task<W, ROPE>(a, ub, b, g, ent, sm, counts, part);
      const int dep = ent.v[5];
      if (dep >= 0) {
        __syncthreads();
        promote_task<W, ROPE>(a, ub, b, g, load_entry(plist, dep), part);
      }
    } else if (ent.v[5] < 0) {
      promote_task<W, ROPE>(a, ub, b, g, ent, part);
    }
    if (task + half < n_tasks) __syncthreads();   // LDS reused by the next task
  }
}

// Copy prompt tokens [tok0, tok1) into the sink slots / recent ring.
__global__ __launch_bounds__(256) void k_pack_tokens(PackArgs a) {
  const Geometry& G = a.g;
  const int g = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  uint8_t* ub = a.base + (int64_t)b * a.L.unit_bytes;
  const int64_t row0 = ((int64_t)b * G.H_kv + g) * a.src_T;
  const int n = (a.tok1 - a.tok0) * kHeadDim;
  for (int i = tid; i < n; i += blockDim.x) {
    const int t = a.tok0 + i / kHeadDim, c = i % kHeadDim;
    uint8_t* dp;
    int tt;
    if (t < G.sink) {
      dp = ub + a.L.sinkp + (int64_t)(t / G.W) * G.fslot_bytes + g * G.fhead_bytes;
      tt = t % G.W;
    } else {
      const int w = (t - G.sink) / G.W;
      dp = ub + a.L.ring + (int64_t)(w % G.NR) * G.fslot_bytes + g * G.fhead_bytes;
      tt = (t - G.sink) % G.W;
    }
    *(uint16_t*)(dp + k_elem_off(G.W, tt, c)) = a.src_k[(row0 + t) * kHeadDim + c];
    *(uint16_t*)(dp + v_elem_off(G.W, tt, c)) = a.src_v[(row0 + t) * kHeadDim + c];
  }
}

// Workgroups per half of the grid: enough for every task of a routing event of
// up to `entries` windows, at most 1024 (larger events loop).
static int migrate_half(const Geometry& g, int entries) {
  int n = entries * g.H_kv * kParts;
  return n < 1 ? 1 : (n > 1024 ? 1024 : n);
}

hipError_t launch_migrate(const MigrateArgs& a, int max_quant, int max_promote, hipStream_t st) {
  const int mx = max_quant > max_promote ? max_quant : max_promote;
  const dim3 grid(2 * migrate_half(a.g, mx), a.g.B, a.n_units);
  if (a.g.rope) {
    if (a.g.W == 32) hipLaunchKernelGGL((k_migrate<32, true>), grid, dim3(kMigrateThreads), 0, st, a);
    else hipLaunchKernelGGL((k_migrate<64, true>), grid, dim3(kMigrateThreads), 0, st, a);
  } else {
    if (a.g.W == 8) hipLaunchKernelGGL((k_migrate<8, false>), grid, dim3(kMigrateThreads), 0, st, a);
    else if (a.g.W == 32) hipLaunchKernelGGL((k_migrate<32, false>), grid, dim3(kMigrateThreads), 0, st, a);
    else hipLaunchKernelGGL((k_migrate<64, false>), grid, dim3(kMigrateThreads), 0, st, a);
  }
  return hipGetLastError();
}
// Registers per lane and LDS bytes per workgroup of the migration kernel a
// geometry launches.
hipError_t migrate_footprint(const Geometry& g, int* vgprs, size_t* lds) {
  const void* k = g.rope ? (g.W == 32 ? reinterpret_cast<const void*>(&k_migrate<32, true>)
                                      : reinterpret_cast<const void*>(&k_migrate<64, true>))
                 : g.W == 8  ? reinterpret_cast<const void*>(&k_migrate<8, false>)
                 : g.W == 32 ? reinterpret_cast<const void*>(&k_migrate<32, false>)
                             : reinterpret_cast<const void*>(&k_migrate<64, false>);
  hipFuncAttributes fa;
  hipError_t e = hipFuncGetAttributes(&fa, k);
  if (e != hipSuccess) return e;
  *vgprs = fa.numRegs;
  *lds = fa.sharedSizeBytes;
  return hipSuccess;
}
hipError_t launch_pack_tokens(const PackArgs& a, hipStream_t st) {
  if (a.tok1 <= a.tok0) return hipSuccess;
  hipLaunchKernelGGL(k_pack_tokens, dim3(a.g.H_kv, a.g.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace qv
