// Tier-aware split-K decode attention and the split merge / window-score pass.
//
// Decode attention of each query head over the accessible tokens (QEvict
// Sec. 3.1): sink and recent tokens and Full windows in bf16, Quantized
// windows as z + s c with the codes expanded in registers.  The pass also
// yields, per (query head, window), the window's softmax mass relative to a
// reference maximum, which the merge turns into the exact attention mass the
// window received and adds, averaged over the query heads, to the window's
// cumulative score (Sec. 3.2, cumulative window score equation).
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
__device__ __forceinline__ u32x4 ld16(const void* p) { return *(const u32x4*)p; }
__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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
// (relative to the new running max) and records the window's (m, l) pair.
template <int TB>
__device__ __forceinline__ void softmax_window(const f32x4 (&acc)[TB], float bias, int ntok,
                                               float scale_log2, int qg, WaveState& st,
                                               float (&p)[TB][4], float* m_out, float* l_out) {
  float x[TB][4];
  float mw = -INFINITY;
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      int t = 16 * tb + 4 * qg + v;
      float y = (acc[tb][v] + bias) * scale_log2;
      y = t < ntok ? y : -INFINITY;
      x[tb][v] = y;
      mw = fmaxf(mw, y);
    }
  mw = fmaxf(mw, __shfl_xor(mw, 16));
  mw = fmaxf(mw, __shfl_xor(mw, 32));
  const float m_new = fmaxf(st.m, mw);
  const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
  float lw = 0.f;
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      p[tb][v] = __builtin_amdgcn_exp2f(x[tb][v] - m_new);
      lw += p[tb][v];
    }
  lw += __shfl_xor(lw, 16);
  lw += __shfl_xor(lw, 32);
  st.l = st.l * alpha + lw;
  st.m = m_new;
  *m_out = m_new;
  *l_out = lw;
  // rescale O rows 4*qg + v by the alpha of head 4*qg + v (held by lane 4*qg + v)
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    float av = __shfl(alpha, 4 * qg + v);
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) st.o[cb][v] *= av;
  }
}

template <int W, int NHS>
__global__ __launch_bounds__(kAttnThreads) void k_attend(AttnArgs a) {
  constexpr int TB = W / 16;
  constexpr int KT = W / 32;
  const Geometry& G = a.g;
  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, qg = lane >> 4;
  const int gqa = G.gqa;

  __shared__ __attribute__((aligned(16))) uint8_t smem[4 * 16 * 130 * 4];
  uint8_t* qlds = smem + wave * 8192;   // [hi/lo][kb][lane] x 16 B

  uint8_t* ub = a.base + (int64_t)b * a.L.unit_bytes;
  const int32_t* counts = (const int32_t*)(ub + a.L.counts);
  const int32_t* icost = (const int32_t*)(ub + a.L.item_cost);
  const int32_t* iref = (const int32_t*)(ub + a.L.item_ref);
  float2* mref = (float2*)(ub + a.L.mref);

  // ---- this split's item range (equal cost) ----
  const int n_fq = counts[CNT_ITEMS];
  const int n_extra = a.n_ring + a.n_sink_items;
  const int n_all = n_fq + n_extra;
  const int cF = G.cost_bf16;
  const int64_t base_cost = icost[n_fq];
  const int64_t total = base_cost + (int64_t)n_extra * cF;
  const int S = G.n_split;
  auto start_cost = [&](int i) -> int64_t {
    return i <= n_fq ? (int64_t)icost[i] : base_cost + (int64_t)(i - n_fq) * cF;
  };
  auto lower = [&](int64_t c) {   // first item whose start cost >= c
    int lo = 0, hi = n_all;
    while (lo < hi) {
      int mid = (lo + hi) >> 1;
      if (start_cost(mid) >= c) hi = mid; else lo = mid + 1;
    }
    return lo;
  };
  const int first = lower((s * total + S - 1) / S);
  const int last = lower(((s + 1) * total + S - 1) / S);

  // ---- query operands ----
  const uint16_t* qbase = a.q + ((int64_t)b * G.H_q + (int64_t)g * gqa) * kHeadDim;
  bf16x8 qop[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    u32x4 v = {0, 0, 0, 0};
    if (r < gqa) v = ld16(qbase + r * kHeadDim + 32 * kb + 8 * qg);
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
#pragma unroll
  for (int i = 0; i < 8; ++i) *(u32x4*)(qlds + (i * 64 + lane) * 16) = (u32x4){0, 0, 0, 0};

  WaveState st;
  st.m = -INFINITY;
  st.l = 0.f;
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) st.o[cb] = (f32x4){0.f, 0.f, 0.f, 0.f};

  const int w_open = (a.T - 1 - G.sink) / W;
  const uint8_t* fpool = ub + a.L.fpool;
  const uint8_t* qpool = ub + a.L.qpool;
  uint8_t* ring = ub + a.L.ring;
  const uint8_t* sinkp = ub + a.L.sinkp;
  const int64_t vbase = (int64_t)W * kHeadDim * 2;

  for (int it = first + wave; it < last; it += 4) {
    int kind = KIND_BF16, ntok = W;
    bool open = false;
    const uint8_t* p;
    if (it < n_fq) {
      const int32_t ref = iref[it];
      kind = ref >> 28;
      const int64_t slot = ref & 0x0FFFFFFF;
      p = kind == KIND_BF16 ? fpool + slot * G.fslot_bytes + g * G.fhead_bytes
                            : qpool + slot * G.qslot_bytes + g * G.qrec_bytes;
    } else if (it < n_fq + a.n_ring) {
      const int w = a.ring_w0 + (it - n_fq);
      p = ring + (int64_t)(w % G.NR) * G.fslot_bytes + g * G.fhead_bytes;
      ntok = min(W, a.T - (G.sink + w * W));
      open = (w == w_open);
    } else {
      const int j = it - n_fq - a.n_ring;
      p = sinkp + (int64_t)j * G.fslot_bytes + g * G.fhead_bytes;
      ntok = min(W, G.sink - j * W);
    }

    f32x4 acc[TB];
    float p_[TB][4];
    float m_w, l_w;
    if (kind == KIND_BF16) {
      u32x4 kc[TB][4], vc[KT][8];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) kc[tb][kb] = ld16(p + ((tb * 4 + kb) * 64 + lane) * 16);
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) vc[kt][cb] = ld16(p + vbase + ((kt * 8 + cb) * 64 + lane) * 16);
      if (ntok < W || open) {
        const int pos = ntok - 1;
        if (open) {   // the token appended this step: use it from the input and store it
          const uint16_t* kn = a.k_new + ((int64_t)b * G.H_kv + g) * kHeadDim;
          const uint16_t* vn = a.v_new + ((int64_t)b * G.H_kv + g) * kHeadDim;
          uint8_t* pw = ring + (p - ring);
#pragma unroll
          for (int tb = 0; tb < TB; ++tb)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
              if (tb == (pos >> 4) && r == (pos & 15)) {
                u32x4 v = ld16(kn + 32 * kb + 8 * qg);
                kc[tb][kb] = v;
                *(u32x4*)(pw + ((tb * 4 + kb) * 64 + lane) * 16) = v;
              }
          int ktp, qp, jp;
          v_tok_pos(pos, &ktp, &qp, &jp);
          if (qg == qp) {
#pragma unroll
            for (int cb = 0; cb < 8; ++cb) {
              const uint16_t val = vn[16 * cb + r];
              *(uint16_t*)(pw + v_elem_off(W, pos, 16 * cb + r)) = val;
#pragma unroll
              for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                  if (kt == ktp && (jp >> 1) == i) {
                    uint32_t wv = vc[kt][cb][i];
                    wv = (jp & 1) ? ((wv & 0x0000FFFFu) | ((uint32_t)val << 16))
                                  : ((wv & 0xFFFF0000u) | val);
                    vc[kt][cb][i] = wv;
                  }
                }
            }
          }
        }
        // tokens past the end of a partial window contribute nothing
#pragma unroll
        for (int kt = 0; kt < KT; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool lo_ok = v_tok(kt, qg, 2 * i) < ntok, hi_ok = v_tok(kt, qg, 2 * i + 1) < ntok;
            const uint32_t mask = (lo_ok ? 0x0000FFFFu : 0u) | (hi_ok ? 0xFFFF0000u : 0u);
#pragma unroll
            for (int cb = 0; cb < 8; ++cb) vc[kt][cb][i] &= mask;
          }
      }
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        acc[tb] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
          acc[tb] = mfma_bf16(__builtin_bit_cast(bf16x8, kc[tb][kb]), qop[kb], acc[tb]);
      }
      softmax_window<TB>(acc, 0.f, ntok, G.scale_log2, qg, st, p_, &m_w, &l_w);
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        bf16x8 pv;
#pragma unroll
        for (int j = 0; j < 8; ++j) pv[j] = (__bf16)p_[2 * kt + (j >> 2)][j & 3];
#pragma unroll
        for (int cb = 0; cb < 8; ++cb)
          st.o[cb] = mfma_bf16(pv, __builtin_bit_cast(bf16x8, vc[kt][cb]), st.o[cb]);
      }
    } else {
      // ---- quantized window: int4 or int2 codes ----
      const bool is4 = kind == KIND_Q4;
      constexpr int NWMAX = W / 4;   // code words per lane at 4 bits
      uint32_t kw[NWMAX], vw[NWMAX];
      const int nld = is4 ? NWMAX / 4 : NWMAX / 8;
#pragma unroll
      for (int m = 0; m < NWMAX / 4; ++m) {
        u32x4 x = {0, 0, 0, 0}, y = {0, 0, 0, 0};
        if (m < nld) {
          x = ld16(p + (m * 64 + lane) * 16);
          y = ld16(p + G.qcodes_bytes + (m * 64 + lane) * 16);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) { kw[4 * m + i] = x[i]; vw[4 * m + i] = y[i]; }
      }
      const uint8_t* mk = p + meta_k_off(G);
      const u32x4 ks8 = ld16(mk + 16 * r);          // scales of channels 8r .. 8r + 7
      const u32x4 kz8 = ld16(mk + 256 + 16 * r);    // zero points
      // value groups of G = W channels (the host enforces G == W)
      constexpr int NG = kHeadDim / W;
      u32x4 vms[KT][NG], vmz[KT][NG];
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int vg = 0; vg < NG; ++vg) {
          const uint8_t* pm = p + meta_v_off(G) + ((kt * 4 + qg) * NG + vg) * 32;
          vms[kt][vg] = ld16(pm);
          vmz[kt][vg] = ld16(pm + 16);
        }

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
          *(u32x4*)(qlds + ((0 * 4 + kb) * 64 + dst) * 16) = __builtin_bit_cast(u32x4, hi8);
          *(u32x4*)(qlds + ((1 * 4 + kb) * 64 + dst) * 16) = __builtin_bit_cast(u32x4, lo8);
        }
        bsum += __shfl_xor(bsum, 1);
        bsum += __shfl_xor(bsum, 2);
        bsum += __shfl_xor(bsum, 4);
        bsum += __shfl_xor(bsum, 8);
        bias_k[k] = bsum;   // q . z of head qg + 4k
      }
      float bias = 0.f;
#pragma unroll
      for (int k = 0; k < NHS; ++k) {
        const float t = __shfl(bias_k[k], 16 * (r & 3));
        if ((r >> 2) == k) bias = t;
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
      softmax_window<TB>(acc, bias, ntok, G.scale_log2, qg, st, p_, &m_w, &l_w);
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
          const u32x4 sv4 = vms[kt][vg], zv4 = vmz[kt][vg];
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
    if (qg == 0 && r < gqa)
      mref[(int64_t)(b * 0 + (g * gqa + r)) * G.max_items + it] = make_float2(m_w, l_w);
  }

  // ---- merge the 4 waves of this split in LDS, write the split partial ----
  __syncthreads();
  float* mo = (float*)smem;   // [wave][head < 16][130]
  if (qg == 0 && r < gqa) {
    mo[(wave * 16 + r) * 130 + 128] = st.m;
    mo[(wave * 16 + r) * 130 + 129] = st.l;
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int row = 4 * qg + v;
    if (row < gqa) {
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) mo[(wave * 16 + row) * 130 + 16 * cb + r] = st.o[cb][v];
    }
  }
  __syncthreads();
  float* part = (float*)(ub + a.L.partial);
  for (int idx = tid; idx < gqa * kHeadDim; idx += kAttnThreads) {
    const int h = idx >> 7, c = idx & 127;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, mo[(w * 16 + h) * 130 + 128]);
    float o = 0.f, L = 0.f;
    if (M > -INFINITY) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float mw = mo[(w * 16 + h) * 130 + 128];
        if (mw > -INFINITY) {
          const float f = __builtin_amdgcn_exp2f(mw - M);
          o += mo[(w * 16 + h) * 130 + c] * f;
          L += mo[(w * 16 + h) * 130 + 129] * f;
        }
      }
    }
    float* pp = part + ((int64_t)(g * gqa + h) * S + s) * (kHeadDim + 2);
    pp[c] = o;
    if (c == 0) {
      pp[kHeadDim] = M;
      pp[kHeadDim + 1] = L;
    }
  }
}

// Split merge (one block per query head) and window-score accumulation
// (mass blocks over the live items): mass_h(w) = 2^(m_w - M_h) l_w / L_h,
// summed over the query heads of each KV group, then over the groups, / H_q.
__global__ __launch_bounds__(256) void k_merge(AttnArgs a) {
  const Geometry& G = a.g;
  const int blk = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  uint8_t* ub = a.base + (int64_t)b * a.L.unit_bytes;
  const int32_t* counts = (const int32_t*)(ub + a.L.counts);
  const float* part = (const float*)(ub + a.L.partial);
  const int S = G.n_split;
  constexpr int PS = kHeadDim + 2;

  if (blk < G.H_q) {
    const int h = blk;
    const float* ph = part + (int64_t)h * S * PS;
    if (tid < kHeadDim) {
      float M = -INFINITY;
      for (int s = 0; s < S; ++s) M = fmaxf(M, ph[s * PS + kHeadDim]);
      float L = 0.f, o = 0.f;
      if (M > -INFINITY) {
        for (int s = 0; s < S; ++s) {
          const float ms = ph[s * PS + kHeadDim];
          if (ms > -INFINITY) {
            const float f = __builtin_amdgcn_exp2f(ms - M);
            L += ph[s * PS + kHeadDim + 1] * f;
            o += ph[s * PS + tid] * f;
          }
        }
      }
      o = L > 0.f ? o / L : 0.f;
      const int64_t oi = ((int64_t)b * G.H_q + h) * kHeadDim + tid;
      if (G.out_bf16) ((uint16_t*)a.out)[oi] = f32_to_bf16_rne(o);
      else ((float*)a.out)[oi] = o;
    }
    return;
  }

  __shared__ float sM[64], sL[64];
  if (tid < G.H_q) {
    const float* ph = part + (int64_t)tid * S * PS;
    float M = -INFINITY;
    for (int s = 0; s < S; ++s) M = fmaxf(M, ph[s * PS + kHeadDim]);
    float L = 0.f;
    if (M > -INFINITY)
      for (int s = 0; s < S; ++s) {
        const float ms = ph[s * PS + kHeadDim];
        if (ms > -INFINITY) L += ph[s * PS + kHeadDim + 1] * __builtin_amdgcn_exp2f(ms - M);
      }
    sM[tid] = M;
    sL[tid] = L;
  }
  __syncthreads();
  const int n_fq = counts[CNT_ITEMS];
  const int n_all = n_fq + a.n_ring + a.n_sink_items;
  const int pos = (blk - G.H_q) * 256 + tid;
  if (pos >= n_all) return;
  const int32_t* iwin = (const int32_t*)(ub + a.L.item_win);
  const int win = pos < n_fq ? iwin[pos] : (pos < n_fq + a.n_ring ? a.ring_w0 + (pos - n_fq) : -1);
  const float2* mref = (const float2*)(ub + a.L.mref);
  float* dbg = (G.flags & 2u) ? (float*)(ub + a.L.dbg_mass) : nullptr;
  float tot = 0.f;
  for (int g = 0; g < G.H_kv; ++g) {
    float sg = 0.f;
    for (int j = 0; j < G.gqa; ++j) {
      const int h = g * G.gqa + j;
      const float2 mr = mref[(int64_t)h * G.max_items + pos];
      const float mass = sL[h] > 0.f ? __builtin_amdgcn_exp2f(mr.x - sM[h]) * mr.y / sL[h] : 0.f;
      sg += mass;
      if (dbg) {
        if (win >= 0) dbg[(int64_t)h * (G.nwc + 1) + win] = mass;
        else atomicAdd(&dbg[(int64_t)h * (G.nwc + 1) + G.nwc], mass);
      }
    }
    tot += sg;
  }
  if (win >= 0) {
    float* score = (float*)(ub + a.L.score);
    score[win] += tot / (float)G.H_q;
  }
}

}  // namespace qv

// ---- launchers -------------------------------------------------------------
namespace qv {
hipError_t launch_attend(const AttnArgs& a, hipStream_t st) {
  dim3 grid(a.g.n_split, a.g.H_kv, a.g.B);
  const int nhs = (a.g.gqa + 3) / 4;
  if (a.g.W == 32) {
    if (nhs == 1) hipLaunchKernelGGL((k_attend<32, 1>), grid, dim3(kAttnThreads), 0, st, a);
    else if (nhs == 2) hipLaunchKernelGGL((k_attend<32, 2>), grid, dim3(kAttnThreads), 0, st, a);
    else hipLaunchKernelGGL((k_attend<32, 4>), grid, dim3(kAttnThreads), 0, st, a);
  } else {
    if (nhs == 1) hipLaunchKernelGGL((k_attend<64, 1>), grid, dim3(kAttnThreads), 0, st, a);
    else if (nhs == 2) hipLaunchKernelGGL((k_attend<64, 2>), grid, dim3(kAttnThreads), 0, st, a);
    else hipLaunchKernelGGL((k_attend<64, 4>), grid, dim3(kAttnThreads), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_merge(const AttnArgs& a, hipStream_t st) {
  const int n_mass = (a.g.max_items + 255) / 256;
  dim3 grid(a.g.H_q + n_mass, a.g.B);
  hipLaunchKernelGGL(k_merge, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}
}  // namespace qv
