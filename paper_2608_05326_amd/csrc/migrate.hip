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

__device__ bool quant_params(float lo, float hi, int nbits, uint16_t* zb, uint16_t* sb) {
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

__device__ int quant_code(float x, double z, double s, int nmax) {
  if (s == 0.0) return 0;
  const double xd = x;
  double c = __builtin_rint((xd - z) / s);
  for (int k = 0; k < 4; ++k) {
    if (xd < z + (c - 0.5) * s) c -= 1.0;
    else if (xd > z + (c + 0.5) * s) c += 1.0;
    else break;
  }
  const bool odd = __builtin_fmod(c, 2.0) != 0.0;
  if (odd && xd == z + (c + 0.5) * s) c += 1.0;
  else if (odd && xd == z + (c - 0.5) * s) c -= 1.0;
  int ci = (int)c;
  return ci < 0 ? 0 : (ci > nmax ? nmax : ci);
}

// Load one KV head of a window into LDS in natural [t][c] layout.
__device__ void load_window(const MigrateArgs& a, uint8_t* ub, int b, int g, int w, int src_kind,
                            int src_idx, uint16_t* sk, uint16_t* sv) {
  const Geometry& G = a.g;
  const int W = G.W, tid = threadIdx.x;
  if (src_kind == SRC_PROMPT) {
    const int64_t row0 = ((int64_t)b * G.H_kv + g) * a.src_T + G.sink + (int64_t)w * W;
    const u32x4* k4 = (const u32x4*)(a.src_k + row0 * kHeadDim);
    const u32x4* v4 = (const u32x4*)(a.src_v + row0 * kHeadDim);
    for (int i = tid; i < W * kHeadDim / 8; i += blockDim.x) {
      ((u32x4*)sk)[i] = k4[i];
      ((u32x4*)sv)[i] = v4[i];
    }
  } else {
    const uint8_t* p = ub + (src_kind == SRC_FSLOT ? a.L.fpool : a.L.ring) +
                       (int64_t)src_idx * G.fslot_bytes + g * G.fhead_bytes;
    // K chunks hold 8 consecutive channels of one token per lane: 16-byte moves
    for (int i = tid; i < W * kHeadDim / 8; i += blockDim.x) {
      const int t = i / 16, c = (i % 16) * 8;
      ((u32x4*)sk)[i] = *(const u32x4*)(p + k_elem_off(t, c));
    }
    for (int i = tid; i < W * kHeadDim; i += blockDim.x) {
      const int t = i >> 7, c = i & 127;
      sv[i] = *(const uint16_t*)(p + v_elem_off(W, t, c));
    }
  }
}

__global__ __launch_bounds__(256) void k_quantize(MigrateArgs a) {
  const Geometry& G = a.g;
  const int b = blockIdx.y, tid = threadIdx.x;
  __shared__ __attribute__((aligned(16))) uint16_t sk[64 * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t sv[64 * kHeadDim];
  __shared__ uint8_t ck[64 * kHeadDim];
  __shared__ uint8_t cv[64 * kHeadDim];
  uint8_t* ub = a.base + (int64_t)b * a.L.unit_bytes;
  int32_t* counts = (int32_t*)(ub + a.L.counts);
  const int32_t* qlist = (const int32_t*)(ub + a.L.qlist);
  const int n = counts[CNT_QUANT];
  const int W = G.W;
  for (int task = blockIdx.x; task < n * G.H_kv; task += gridDim.x) {
    const int e = task / G.H_kv, g = task % G.H_kv;
    const int32_t* ent = qlist + e * kQEntry;
    const int w = ent[0], src_kind = ent[1], src_idx = ent[2], dst = ent[3], nb = ent[4];
    load_window(a, ub, b, g, w, src_kind, src_idx, sk, sv);
    __syncthreads();
    uint8_t* rec = ub + a.L.qpool + (int64_t)dst * G.qslot_bytes + g * G.qrec_bytes;
    const int nmax = (1 << nb) - 1;
    if (tid < kHeadDim) {
      // key group: channel tid across the window's tokens
      const int c = tid;
      float lo = INFINITY, hi = -INFINITY;
      for (int t = 0; t < W; ++t) {
        const float x = bf16_to_f32(sk[t * kHeadDim + c]);
        lo = fminf(lo, x);
        hi = fmaxf(hi, x);
      }
      uint16_t zb = 0, sb = 0;
      if (!quant_params(lo, hi, nb, &zb, &sb)) set_error(counts, ERR_RANGE);
      const double z = fp16_bits_to_f64(zb), s = fp16_bits_to_f64(sb);
      for (int t = 0; t < W; ++t)
        ck[t * kHeadDim + c] = (uint8_t)quant_code(bf16_to_f32(sk[t * kHeadDim + c]), z, s, nmax);
      uint16_t* mk = (uint16_t*)(rec + meta_k_off(G));
      mk[c] = sb;
      mk[kHeadDim + c] = zb;
    } else {
      // value groups: token t, channels vg*G .. vg*G + G - 1
      const int ng = kHeadDim / G.G;
      for (int idx = tid - kHeadDim; idx < W * ng; idx += blockDim.x - kHeadDim) {
        const int t = idx / ng, vg = idx % ng;
        const uint16_t* row = sv + t * kHeadDim + vg * G.G;
        float lo = INFINITY, hi = -INFINITY;
        for (int i = 0; i < G.G; ++i) {
          const float x = bf16_to_f32(row[i]);
          lo = fminf(lo, x);
          hi = fmaxf(hi, x);
        }
        uint16_t zb = 0, sb = 0;
        if (!quant_params(lo, hi, nb, &zb, &sb)) set_error(counts, ERR_RANGE);
        const double z = fp16_bits_to_f64(zb), s = fp16_bits_to_f64(sb);
        for (int i = 0; i < G.G; ++i)
          cv[t * kHeadDim + vg * G.G + i] = (uint8_t)quant_code(bf16_to_f32(row[i]), z, s, nmax);
        uint16_t* mv = (uint16_t*)(rec + meta_v_elem(G, t, vg));
        mv[0] = sb;
        mv[8] = zb;
      }
    }
    __syncthreads();
    // pack codes: storage word (m, lane, comp) holds 4/nb entries of 8 codes
    const int words = W * kHeadDim * nb / 32;   // per code area
    const int per = 4 / nb;
    for (int sp = tid; sp < words; sp += blockDim.x) {
      const int m = sp >> 8, L = (sp >> 2) & 63, comp = sp & 3;
      const int word = m * 4 + comp;
      uint32_t wk = 0, wv = 0;
      for (int ee = 0; ee < per; ++ee) {
        const int ent_idx = word * per + ee;
        for (int j = 0; j < 8; ++j) {
          const int sh = (j & 1) * 16 + nb * (4 * ee + (j >> 1));
          // key entry (tb, kb): token 16 tb + (L & 15), channel 32 kb + 8 (L >> 4) + j
          const int tk = 16 * (ent_idx >> 2) + (L & 15);
          const int chk = 32 * (ent_idx & 3) + 8 * (L >> 4) + j;
          wk |= (uint32_t)ck[tk * kHeadDim + chk] << sh;
          // value entry (kt, cb): token tok(kt, L >> 4, j), channel 16 cb + (L & 15)
          const int tv = v_tok(ent_idx >> 3, L >> 4, j);
          const int chv = 16 * (ent_idx & 7) + (L & 15);
          wv |= (uint32_t)cv[tv * kHeadDim + chv] << sh;
        }
      }
      *(uint32_t*)(rec + (int64_t)sp * 4) = wk;
      *(uint32_t*)(rec + G.qcodes_bytes + (int64_t)sp * 4) = wv;
    }
    __syncthreads();
  }
}

__device__ __forceinline__ int read_code(const uint8_t* area, int nb, int e, int L, int j) {
  int64_t off;
  int sh;
  code_loc(nb, e, L, j, &off, &sh);
  return (int)((*(const uint32_t*)(area + off) >> sh) & ((1u << nb) - 1));
}

__global__ __launch_bounds__(256) void k_promote(MigrateArgs a) {
  const Geometry& G = a.g;
  const int b = blockIdx.y, tid = threadIdx.x;
  uint8_t* ub = a.base + (int64_t)b * a.L.unit_bytes;
  int32_t* counts = (int32_t*)(ub + a.L.counts);
  const int32_t* plist = (const int32_t*)(ub + a.L.plist);
  const int n = counts[CNT_PROMOTE];
  const int W = G.W;
  for (int task = blockIdx.x; task < n * G.H_kv; task += gridDim.x) {
    const int e = task / G.H_kv, g = task % G.H_kv;
    const int32_t* ent = plist + e * kQEntry;
    const int w = ent[0], src_kind = ent[1], src_idx = ent[2], dst = ent[3], nb = ent[4];
    uint8_t* dp = ub + a.L.fpool + (int64_t)dst * G.fslot_bytes + g * G.fhead_bytes;
    if (src_kind == SRC_RING) {
      const u32x4* sp = (const u32x4*)(ub + a.L.ring + (int64_t)src_idx * G.fslot_bytes +
                                       g * G.fhead_bytes);
      for (int i = tid; i < G.fhead_bytes / 16; i += blockDim.x) ((u32x4*)dp)[i] = sp[i];
    } else if (src_kind == SRC_PROMPT) {
      const int64_t row0 = ((int64_t)b * G.H_kv + g) * a.src_T + G.sink + (int64_t)w * W;
      const uint16_t* ks = a.src_k + row0 * kHeadDim;
      const uint16_t* vs = a.src_v + row0 * kHeadDim;
      for (int i = tid; i < W * kHeadDim / 8; i += blockDim.x) {
        const int t = i / 16, c = (i % 16) * 8;
        *(u32x4*)(dp + k_elem_off(t, c)) = *(const u32x4*)(ks + t * kHeadDim + c);
      }
      for (int i = tid; i < W * kHeadDim; i += blockDim.x) {
        const int t = i >> 7, c = i & 127;
        *(uint16_t*)(dp + v_elem_off(W, t, c)) = vs[t * kHeadDim + c];
      }
    } else {   // SRC_QSLOT: exact dequantization, single rounding to bf16
      const uint8_t* rec = ub + a.L.qpool + (int64_t)src_idx * G.qslot_bytes + g * G.qrec_bytes;
      const uint16_t* mk = (const uint16_t*)(rec + meta_k_off(G));
      for (int i = tid; i < W * kHeadDim; i += blockDim.x) {
        const int t = i >> 7, c = i & 127;
        int ee, L, j;
        k_code_pos(t, c, &ee, &L, &j);
        const int code = read_code(rec, nb, ee, L, j);
        const double x = fp16_bits_to_f64(mk[kHeadDim + c]) + fp16_bits_to_f64(mk[c]) * code;
        *(uint16_t*)(dp + k_elem_off(t, c)) = f64_to_bf16_rne(x);
        v_code_pos(t, c, &ee, &L, &j);
        const int cvv = read_code(rec + G.qcodes_bytes, nb, ee, L, j);
        const uint16_t* mv = (const uint16_t*)(rec + meta_v_elem(G, t, c / G.G));
        const double y = fp16_bits_to_f64(mv[8]) + fp16_bits_to_f64(mv[0]) * cvv;
        *(uint16_t*)(dp + v_elem_off(W, t, c)) = f64_to_bf16_rne(y);
      }
    }
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
    *(uint16_t*)(dp + k_elem_off(tt, c)) = a.src_k[(row0 + t) * kHeadDim + c];
    *(uint16_t*)(dp + v_elem_off(G.W, tt, c)) = a.src_v[(row0 + t) * kHeadDim + c];
  }
}

static int migrate_blocks(const Geometry& g, int max_entries) {
  int n = max_entries * g.H_kv;
  return n < 1 ? 1 : (n > 256 ? 256 : n);
}

hipError_t launch_quantize(const MigrateArgs& a, int max_entries, hipStream_t st) {
  hipLaunchKernelGGL(k_quantize, dim3(migrate_blocks(a.g, max_entries), a.g.B), dim3(256), 0, st, a);
  return hipGetLastError();
}
hipError_t launch_promote(const MigrateArgs& a, int max_entries, hipStream_t st) {
  hipLaunchKernelGGL(k_promote, dim3(migrate_blocks(a.g, max_entries), a.g.B), dim3(256), 0, st, a);
  return hipGetLastError();
}
hipError_t launch_pack_tokens(const PackArgs& a, hipStream_t st) {
  if (a.tok1 <= a.tok0) return hipSuccess;
  hipLaunchKernelGGL(k_pack_tokens, dim3(a.g.H_kv, a.g.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace qv
