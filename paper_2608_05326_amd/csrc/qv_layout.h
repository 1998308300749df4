// Device memory layout of the tiered KV cache (shared by host runtime and kernels).
//
// Everything lives in one caller-provided workspace:
//   [header][unit 0][unit 1]...   unit u = layer * B + seq
// Each unit block holds the bf16 window pool (Full tier), the recent-region
// ring, the sink slots, the quantized-record pool (Quantized tier plus dormant
// ledgers), the per-window state arrays, the live-window list, the migration
// work lists and the split-K partials of that (sequence, layer).
//
// bf16 window slot, one KV head (W tokens x 128 channels, K then V):
//   K part: chunk (tb, kb), tb = t/16, kb = c/32, 1 KiB each; lane L = 16q + r
//           holds K[16 tb + r][32 kb + 8 q + j], j = 0..7 (16 bytes at 16 L).
//           This is the A operand of a 16x16x32 MFMA with tokens as rows.
//   V part: chunk (kt, cb), kt = t/32, cb = c/16; lane L = 16q + r holds
//           V[tok(kt, q, j)][16 cb + r], j = 0..7, with
//           tok(kt, q, j) = 32 kt + 16 (j/4) + 4 q + (j%4):
//           the B operand of the P.V MFMA whose k index matches the row layout
//           of the QK^T accumulator, so probabilities never move between lanes.
// Quantized record, one KV head: [K codes][V codes][K meta][V meta]
//   codes use the same (entry, lane) positions as the bf16 chunks, 8 codes per
//   (entry, lane); code j = 2i + o sits at bit 16 o + b (4 e' + i), e' = the
//   entry's position inside its 32-bit word (int4: one entry per word, int2:
//   two), so an AND with 0x000F000F / 0x00030003 after a shift yields two codes
//   in the two fp16 halves of a register.
//   K meta: fp16 scale[128] then zero[128] (one key group per channel per window).
//   V meta: per (kt, q, value group g): fp16 scale[8] then zero[8] for the 8
//           tokens tok(kt, q, 0..7).
//
// 8-token windows (values in groups of G = 32 channels) use their own chunks:
//   bf16 K: chunk kb (channels 32 kb ..), 512 B: lane L = 16q + r, r < 8, holds
//           K[r][32 kb + 8 q + j] at ((kb * 4 + q) * 8 + r) * 16 + 2 j -- rows 0..7
//           of the QK^T A operand (rows 8..15 of the tile stay empty);
//   bf16 V: chunk cp (channel blocks 2 cp and 2 cp + 1), 512 B: lane L = 16q + r,
//           q < 2, holds V[4 q + j][16 (2 cp + e) + r] at
//           ((cp * 2 + q) * 16 + r) * 16 + 8 e + 2 j -- the B operand (tokens
//           4 q .. 4 q + 3) of a 16x16x16 P.V MFMA for channel block 2 cp + e;
//   K codes: lane (q, r < 8) holds the 32 codes of token r, channels 32 kb + 8 q + j,
//           in 16 B (int4: word kb) or 8 B (int2: word kb / 2, entry kb % 2) at
//           (q * 8 + r) * (16 or 8); code j = 2i + o at bit 16 o + b (4 e' + i);
//   V codes: lane (q < 2, r) holds the codes of tokens 4 q + j, channel blocks
//           cb = 0..7 (channel 16 cb + r): word cp (int4) or word cp / 2, entry
//           cp % 2 (int2) holds, at position i' = 2 (cb % 2) + j / 2, o = j % 2,
//           the code of token 4 q + j of block cb; lane offset (q * 16 + r) * (16 or 8);
//   K meta as above; V meta: per (q < 2, value group g < 4): fp16 scale[4] then
//           zero[4] for tokens 4 q .. 4 q + 3 at (q * 4 + g) * 16.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define QV_HD __host__ __device__ inline
#else
#define QV_HD inline
#endif

namespace qv {

constexpr int kHeadDim = 128;
constexpr int kMaxGqa = 16;
constexpr int kMaxCand = 4096;      // candidates per routing event (one workgroup sorts them)
constexpr int kAttnThreads = 256;
constexpr int kRetierThreads = 1024;

// tier codes stored on the device (same numbers as the ABI)
enum : int8_t { T_UNUSED = 0, T_OPEN = 1, T_FULL = 2, T_QUANT = 3, T_EVICTED = 4 };
enum : int8_t { L_NONE = 0, L_ACTIVE = 1, L_DORMANT = 2 };
// live-item kinds
enum : int32_t { KIND_BF16 = 0, KIND_Q4 = 1, KIND_Q2 = 2 };
// item_aux of a live item: -1, or the quantized slot of the window's ledger
// (dormant for a Full item, active for a Quantized one) with its bit width:
// aux = qslot | (bits << 28)
// per-unit counters
// (CNT_COST: summed split-balancing cost of the live list, item_cost[CNT_ITEMS];
//  CNT_PLAN_T0 + 2j .. CNT_PLAN_T1 + 2j: the sequence lengths split plan slot j
//  holds for, first > last when it holds none)
enum : int32_t { CNT_ITEMS = 0, CNT_QUANT = 1, CNT_PROMOTE = 2, CNT_ERROR = 3, CNT_BYTES_LO = 4,
                 CNT_COST = 5, CNT_PLAN_T0 = 6, CNT_PLAN_T1 = 7, CNT_N = 16 };
// split plan record: first item, end item, list refs of the first kPlanRefs items.
// A plan depends on the live list and on the number of recent-region and sink
// windows after it, which grows by one each time a window starts; the list only
// changes at a routing event, so kPlanSlots plans (one per such count) cover the
// steps up to the next event.
constexpr int kPlanRefs = 6;
constexpr int kPlanRec = 2 + kPlanRefs;
constexpr int kPlanSlots = 2;
// device error bits
enum : int32_t { ERR_NONFINITE = 1, ERR_POOL = 2, ERR_RANGE = 4, ERR_CAND = 8, ERR_GATE = 16 };
// stats slots (same order as qevict_retier_stats)
enum : int32_t { ST_PROMO = 0, ST_ADMIT = 1, ST_FIRSTQ = 2, ST_REACT = 3, ST_EVICT = 4,
                 ST_NF = 5, ST_NQ4 = 6, ST_NQ2 = 7, ST_N = 8 };
// work-list sources
enum : int32_t { SRC_FSLOT = 0, SRC_RING = 1, SRC_PROMPT = 2, SRC_QSLOT = 3 };
// ints per work-list entry: win, src_kind, src_idx, dst, bits, dep; dep pairs a
// quantization that reads a bf16 slot with the promotion / admission that
// writes the same slot (index of the other list's entry, or -1)
constexpr int kQEntry = 6;
// spare bf16 pool slots beyond K_f (fewer when the owner tables would not fit)
constexpr int kSpareFull = 8;
// sink windows per sequence (keeps the attention split costs in 32 bits)
constexpr int kMaxSinkWindows = 64;
// bytes of the fixed per-device scratch of the allocation-free initial-score call
constexpr int64_t kStaticObsScratchBytes = 16LL << 20;

constexpr int kScorePnorm = 3;   // score_mode of the attention p-norm ranking

struct Geometry {
  int32_t B, H_q, H_kv, gqa, d, W, G;
  int32_t bits_cfg;     // 4, 2 or 42
  int32_t qbits_max;    // 4 or 2: code area size of a record
  int32_t K_f, K_q, n_qslots;
  int32_t n_fslots;     // bf16 pool slots: K_f plus spares (a promotion then takes a slot
                        // that was free before the event, not one vacated in it)
  int32_t NR, NS;       // ring slots, sink slots
  int32_t sink, recent;
  int32_t nwc;          // window capacity per unit
  int32_t max_items;    // Full + Quantized + ring + sink items
  int32_t max_fq;       // K_f + K_q
  int32_t n_split;
  int32_t out_bf16;
  uint32_t flags;
  int32_t score_mode;   // window ranking function (cumulative, decayed, key norm, p-norm)
  const float* rope;    // RoPE table [max_context][64] (cos, sin) pairs; null without RoPE
  float scale_log2;     // softmax scale * log2(e)
  int64_t fhead_bytes;  // one KV head of a bf16 slot: W*d*2 (K) + W*d*2 (V)
  int64_t fslot_bytes;  // H_kv * fhead_bytes
  int64_t qcodes_bytes; // W*d*qbits_max/8, one of K or V
  int64_t qrec_bytes;   // one KV head of a quantized record
  int64_t qslot_bytes;  // H_kv * qrec_bytes
  int32_t cost_bf16, cost_q4, cost_q2;   // split balancing weights per item
};

struct UnitLayout {
  int64_t unit_bytes;
  int64_t fpool, ring, sinkp, qpool;
  int64_t tier, ledger, bits, fslot, qslot, score;
  int64_t fowner, qowner;
  int64_t item_win, item_ref, item_cost, item_aux, item_score;
  int64_t qlist, plist, counts, stats;
  int64_t partial, pml, mref, dbg_mass;
  int64_t plan;         // per (split, wave): first item, end item, refs of its first kPlanRefs items
  int64_t pnorm;        // p-norm ranking only: per window {sum of completed periods' u^p, running u}
};

QV_HD int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// ---- bf16 slot offsets (bytes inside one KV head block) ---------------------
QV_HD int64_t k_elem_off(int W, int t, int c) {
  const int kb = c >> 5, q = (c >> 3) & 3, j = c & 7;
  if (W == 8) return ((int64_t)((kb * 4 + q) * 8 + t) * 16) + j * 2;
  const int tb = t >> 4, r = t & 15;
  return ((int64_t)((tb * 4 + kb) * 64 + q * 16 + r) * 16) + j * 2;
}
QV_HD void v_tok_pos(int t, int* kt, int* q, int* j) {
  int tt = t & 31;
  *kt = t >> 5;
  *q = (tt & 15) >> 2;
  *j = ((tt >> 4) << 2) | (tt & 3);
}
QV_HD int v_tok(int kt, int q, int j) { return 32 * kt + 16 * (j >> 2) + 4 * q + (j & 3); }
QV_HD int64_t v_elem_off(int W, int t, int c) {
  const int cb = c >> 4, r = c & 15;
  if (W == 8) {
    const int q = t >> 2, j = t & 3, cp = cb >> 1, e = cb & 1;
    return (int64_t)W * kHeadDim * 2 + ((int64_t)((cp * 2 + q) * 16 + r) * 16) + 8 * e + 2 * j;
  }
  int kt, q, j;
  v_tok_pos(t, &kt, &q, &j);
  return (int64_t)W * kHeadDim * 2 + ((int64_t)((kt * 8 + cb) * 64 + q * 16 + r) * 16) + j * 2;
}

// ---- quantized record offsets -----------------------------------------------
// location of code (entry e, lane L, element j) of one code area
QV_HD void code_loc(int bits, int e, int L, int j, int64_t* byte_off, int* shift) {
  int per_word = 4 / bits;                 // entries in one 32-bit word: int4 -> 1, int2 -> 2
  int word = e / per_word, ee = e % per_word;
  int i = j >> 1, o = j & 1;
  *byte_off = ((int64_t)((word >> 2) * 64 + L) * 16) + (word & 3) * 4;
  *shift = o * 16 + bits * (4 * ee + i);
}
QV_HD void k_code_pos(int t, int c, int* e, int* L, int* j) {
  *e = (t >> 4) * 4 + (c >> 5);
  *L = ((c >> 3) & 3) * 16 + (t & 15);
  *j = c & 7;
}
QV_HD void v_code_pos(int t, int c, int* e, int* L, int* j) {
  int kt, q, jj;
  v_tok_pos(t, &kt, &q, &jj);
  *e = kt * 8 + (c >> 4);
  *L = q * 16 + (c & 15);
  *j = jj;
}
// 8-token windows: byte offset inside a code area and bit shift of the code of
// token t, channel c (area 0 keys, 1 values)
QV_HD void code_loc8(int bits, int area, int t, int c, int64_t* byte_off, int* shift) {
  const int lb = bits == 4 ? 16 : 8;   // bytes of codes per lane
  if (area == 0) {
    const int kb = c >> 5, q = (c >> 3) & 3, j = c & 7;
    const int word = bits == 4 ? kb : kb >> 1, ee = bits == 4 ? 0 : kb & 1;
    *byte_off = (int64_t)(q * 8 + t) * lb + 4 * word;
    *shift = (j & 1) * 16 + bits * (4 * ee + (j >> 1));
  } else {
    const int q = t >> 2, j = t & 3, cb = c >> 4, r = c & 15, cp = cb >> 1;
    const int word = bits == 4 ? cp : cp >> 1, ee = bits == 4 ? 0 : cp & 1;
    const int i = 2 * (cb & 1) + (j >> 1);
    *byte_off = (int64_t)(q * 16 + r) * lb + 4 * word;
    *shift = (j & 1) * 16 + bits * (4 * ee + i);
  }
}
// meta offsets inside a record (after the two code areas)
QV_HD int64_t meta_k_off(const Geometry& g) { return 2 * g.qcodes_bytes; }
QV_HD int64_t meta_v_off(const Geometry& g) { return 2 * g.qcodes_bytes + 4 * kHeadDim; }
// byte offset of the V scale of token t, value group vg; its zero point follows
// meta_v_zero_delta bytes later
QV_HD int64_t meta_v_elem(const Geometry& g, int t, int vg) {
  if (g.W == 8) return meta_v_off(g) + (int64_t)(((t >> 2) * 4 + vg) * 16) + (t & 3) * 2;
  int kt, q, j;
  v_tok_pos(t, &kt, &q, &j);
  int ng = kHeadDim / g.G;
  return meta_v_off(g) + ((int64_t)((kt * 4 + q) * ng + vg) * 32) + j * 2;
}
QV_HD int meta_v_zero_delta(const Geometry& g) { return g.W == 8 ? 8 : 16; }

QV_HD int item_cost(const Geometry& g, int kind) {
  return kind == KIND_BF16 ? g.cost_bf16 : (kind == KIND_Q4 ? g.cost_q4 : g.cost_q2);
}

}  // namespace qv
