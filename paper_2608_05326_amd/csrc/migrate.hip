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

// Round-half-even code of x: an fp32 estimate of (x - z) / s, then the exact
// decision against the two neighbouring half-step boundaries z + (c +- 1/2) s
// (exact in float64: fp16 operands, |c| <= 16).  No division per element.
__device__ __forceinline__ int quant_code(float x, float zf, float inv_s, double z, double s,
                                          int nmax) {
  if (s == 0.0) return 0;
  float c0 = rintf((x - zf) * inv_s);
  c0 = fminf(fmaxf(c0, 0.f), (float)nmax);
  int c = (int)c0;
  const double xd = x;
  for (int k = 0; k < 2; ++k) {
    const double hi = z + ((double)c + 0.5) * s, lo = z + ((double)c - 0.5) * s;
    if ((xd > hi || (xd == hi && (c & 1))) && c < nmax) {
      ++c;
    } else if ((xd < lo || (xd == lo && (c & 1))) && c > 0) {
      --c;
    } else {
      break;
    }
  }
  return c;
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
    const uint8_t* pv = p + (int64_t)W * kHeadDim * 2;
    // K chunk (tb, kb), lane 16q + r: token 16 tb + r, channels 32 kb + 8 q .. + 7
    // V chunk (kt, cb), lane 16q + r: tokens tok(kt, q, 0..7), channel 16 cb + r
    for (int i = tid; i < W * kHeadDim / 8; i += blockDim.x) {
      const int chunk = i >> 6, L = i & 63, q = L >> 4, r = L & 15;
      const u32x4 kx = *(const u32x4*)(p + (int64_t)i * 16);
      const u32x4 vx = *(const u32x4*)(pv + (int64_t)i * 16);
      *(u32x4*)(sk + (16 * (chunk >> 2) + r) * kHeadDim + 32 * (chunk & 3) + 8 * q) = kx;
      const int kt = chunk >> 3, c = 16 * (chunk & 7) + r;
      const uint32_t v0 = vx[0], v1 = vx[1], v2 = vx[2], v3 = vx[3];
      const uint32_t vw[4] = {v0, v1, v2, v3};
#pragma unroll
      for (int j = 0; j < 8; ++j)
        sv[v_tok(kt, q, j) * kHeadDim + c] = (uint16_t)(vw[j >> 1] >> (16 * (j & 1)));
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
      const float zf = (float)z, inv_s = s > 0.0 ? 1.f / (float)s : 0.f;
      for (int t = 0; t < W; ++t)
        ck[t * kHeadDim + c] =
            (uint8_t)quant_code(bf16_to_f32(sk[t * kHeadDim + c]), zf, inv_s, z, s, nmax);
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
        const float zf = (float)z, inv_s = s > 0.0 ? 1.f / (float)s : 0.f;
        for (int i = 0; i < G.G; ++i)
          cv[t * kHeadDim + vg * G.G + i] =
              (uint8_t)quant_code(bf16_to_f32(row[i]), zf, inv_s, z, s, nmax);
        uint16_t* mv = (uint16_t*)(rec + meta_v_elem(G, t, vg));
        mv[0] = sb;
        mv[8] = zb;
      }
    }
    __syncthreads();
    // pack: thread (area, block m, lane L) writes the 16-byte block of words 4m .. 4m + 3 of
    // lane L; word wd holds entries wd * per + ee (per = 4 / nb), 8 codes each
    const int nblk = W * nb / 64;
    const int per = 4 / nb;
    for (int tk = tid; tk < 2 * nblk * 64; tk += blockDim.x) {
      const int area = tk / (nblk * 64), m = (tk >> 6) % nblk, L = tk & 63;
      const int q = L >> 4, r = L & 15;
      uint32_t wv[4];
#pragma unroll
      for (int comp = 0; comp < 4; ++comp) {
        uint32_t wd = 0;
        for (int ee = 0; ee < per; ++ee) {
          const int ei = (m * 4 + comp) * per + ee;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int sh = (j & 1) * 16 + nb * (4 * ee + (j >> 1));
            uint32_t code;
            if (area == 0)   // key entry (tb, kb): token 16 tb + r, channel 32 kb + 8 q + j
              code = ck[(16 * (ei >> 2) + r) * kHeadDim + 32 * (ei & 3) + 8 * q + j];
            else             // value entry (kt, cb): token tok(kt, q, j), channel 16 cb + r
              code = cv[v_tok(ei >> 3, q, j) * kHeadDim + 16 * (ei & 7) + r];
            wd |= code << sh;
          }
        }
        wv[comp] = wd;
      }
      *(u32x4*)(rec + area * G.qcodes_bytes + ((int64_t)m * 64 + L) * 16) =
          (u32x4){wv[0], wv[1], wv[2], wv[3]};
    }
    __syncthreads();
  }
}

// 8 bf16 values z_j + s_j c_j (exact in float64, one rounding) packed for a 16-byte store
__device__ __forceinline__ u32x4 dequant8(uint32_t wd, int shift0, int nb, u32x4 s8, u32x4 z8) {
  const uint32_t mask = (1u << nb) - 1u;
  const uint32_t sw[4] = {s8[0], s8[1], s8[2], s8[3]};
  const uint32_t zw[4] = {z8[0], z8[1], z8[2], z8[3]};
  uint32_t outw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t pair = 0;
#pragma unroll
    for (int o = 0; o < 2; ++o) {
      const int j = 2 * i + o;
      const uint32_t code = (wd >> (o * 16 + shift0 + nb * i)) & mask;
      const double sj = fp16_bits_to_f64((uint16_t)(sw[i] >> (16 * o)));
      const double zj = fp16_bits_to_f64((uint16_t)(zw[i] >> (16 * o)));
      pair |= (uint32_t)f64_to_bf16_rne(zj + sj * (double)code) << (16 * o);
      (void)j;
    }
    outw[i] = pair;
  }
  return (u32x4){outw[0], outw[1], outw[2], outw[3]};
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
    } else {
      // SRC_QSLOT: thread (area, block m, lane L) expands the entries held by the 16-byte
      // code block m of lane L straight into the bf16 chunks at the same (entry, lane)
      const uint8_t* rec = ub + a.L.qpool + (int64_t)src_idx * G.qslot_bytes + g * G.qrec_bytes;
      const int nblk = W * nb / 64;
      const int per = 4 / nb;
      const int ng = kHeadDim / G.G;
      for (int tk = tid; tk < 2 * nblk * 64; tk += blockDim.x) {
        const int area = tk / (nblk * 64), m = (tk >> 6) % nblk, L = tk & 63;
        const int q = L >> 4, r = L & 15;
        const u32x4 blk = *(const u32x4*)(rec + area * G.qcodes_bytes + ((int64_t)m * 64 + L) * 16);
        const uint32_t bw[4] = {blk[0], blk[1], blk[2], blk[3]};
        for (int comp = 0; comp < 4; ++comp) {
          for (int ee = 0; ee < per; ++ee) {
            const int ei = (m * 4 + comp) * per + ee;
            u32x4 s8, z8;
            int64_t off;
            if (area == 0) {   // key entry (tb, kb): channels 32 kb + 8 q .. + 7 of token 16 tb + r
              const int c0 = 32 * (ei & 3) + 8 * q;
              s8 = *(const u32x4*)(rec + meta_k_off(G) + 2 * c0);
              z8 = *(const u32x4*)(rec + meta_k_off(G) + 2 * kHeadDim + 2 * c0);
              off = ((int64_t)ei * 64 + L) * 16;
            } else {           // value entry (kt, cb): tokens tok(kt, q, 0..7) of channel 16 cb + r
              const int kt = ei >> 3, c = 16 * (ei & 7) + r;
              const uint8_t* pm = rec + meta_v_off(G) + ((kt * 4 + q) * ng + c / G.G) * 32;
              s8 = *(const u32x4*)pm;
              z8 = *(const u32x4*)(pm + 16);
              off = (int64_t)W * kHeadDim * 2 + ((int64_t)ei * 64 + L) * 16;
            }
            *(u32x4*)(dp + off) = dequant8(bw[comp], 4 * nb * ee, nb, s8, z8);
          }
        }
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
