// Decode attention over the paged KV cache (one or a few queries per sequence).
//
// "KVCache Storage Analysis": decode is memory-bound, its cost follows the KV
// bytes read; SWA layers read at most W keys from the per-sequence ring, FULL
// layers read the whole context.
//
// Work: an SWA layer (or a FULL layer short enough for one pass) has one item
// per (sequence, KV head, group of up to 16 query heads of that KV head)
// covering every visible key; a workgroup of four waves shares the item. A
// FULL layer walks all (sequence, head group) segments of 32-key chunks, in
// that order, cut into equal spans, one per wave the device holds at once
// (stream-K): every wave gets the same number of chunks whatever the mix of
// context lengths, and crosses segment boundaries inside its span.
//
// Per item the wave walks 32-key chunks and runs both products on the bf16
// matrix cores with the GQA query heads as the 16 MFMA columns:
//   S^T[key][head]  = K[key][:] . Q[head][:]        (K slabs straight from HBM)
//   O^T[d][head]   += V^T[d][key] . P^T[key][head]   (V pages hold [D][32] blocks)
// The 32 keys of a chunk are assigned to MFMA rows so that the score tile comes
// out with each lane holding 8 consecutive keys of one head, which is exactly
// the lane layout the PV product needs for P^T: no shuffle between the two; the
// K pool stores each 32-key block in that row order, so every K load
// instruction reads one contiguous 1 KiB (and every V load as well).
// Softmax is online per chunk in fp32 (exp2 with scale*log2(e) folded in).
// FULL split spans run one wave per SIMD with two whole chunks of loads in
// flight while a third is computed (fewer, deeper streams read HBM faster
// than more, shallower ones). Whole-range items: the K loads of chunk c+1 are
// in flight while chunk c's softmax and PV run, its V loads while chunk c+1's
// QK^T runs. A segment cut by span boundaries
// gets fp32 (o, log2 sum-exp) partials that a second kernel merges; a segment
// inside one span, and a whole-range item, is written as bf16 directly.
// In a decode step with its append ("KVCache Dual-Pool Design": the step's
// token goes to its slot), the split spans of one-page chunks also store the
// token: the wave holding a segment's last chunk takes the token's key from
// the input rows and writes them to the slot.
#include <atomic>
#include <cfloat>

#include "hswa_common.h"
#include "hswa_launch.h"

namespace hswa {
namespace {

// KV bytes are read once per call: non-temporal loads keep them from
// displacing reusable lines in L2 and the memory-side cache.
__device__ __forceinline__ u32x4 ldnt128(const void *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

constexpr int kChunk = 32;
constexpr int kCols = 16;  // query heads per item (MFMA columns)
constexpr int kMergeThreads = 256;
constexpr float kRescaleLog2 = 8.f;  // lazy raise threshold of the running maximum (exp2 units)

// Per-wave copy of a window of the block table: lane i holds the physical page
// of logical page lp0 + i (-1 if outside the range or not a valid page id), so
// page ids are read with v_readlane instead of a dependent global load per chunk.
struct LaneTable {
  int page;
  int lp0;
};

__device__ __forceinline__ void load_lane_table(LaneTable &t, const PoolView &pv, int b, int lp0, int last_lp,
                                                int lane) {
  t.lp0 = lp0;
  const int lp = lp0 + lane;
  int page = -1;
  if (lp <= last_lp) {
    const int e = pv.ring > 0 ? lp % pv.ring : lp;
    const int64_t v = pv.table[(int64_t)b * pv.stride + e];
    page = (v >= 0 && v < pv.num_pages) ? (int)v : -1;
  }
  t.page = page;
}

// Bits i (0 .. 7) of the keys k0 + i inside [lo, hi].
__device__ __forceinline__ uint32_t key_bits(int k0, int lo, int hi) {
  const int a = min(max(lo - k0, 0), 8);
  const int z = min(max(hi - k0 + 1, 0), 8);
  return ((1u << z) - 1u) & ~((1u << a) - 1u);
}

// 32-key chunks of sequence bb's context (0 past the batch or for an empty context).
__device__ __forceinline__ int seq_chunks(const DecodeParams &p, int bb) {
  if (bb >= p.ns) return 0;
  const int c = min(p.ctx_lens[bb], p.max_ctx);
  return c >= 1 ? (c + kChunk - 1) / kChunk : 0;
}

__device__ __forceinline__ int64_t wave_sum64(int v) {
  int64_t s = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) s += __shfl_xor(s, off, kWave);
  return s;
}

// A value every lane holds alike, marked wave-uniform (scalar registers).
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int64_t uni64(int64_t v) {
  const uint64_t x = (uint64_t)v;
  return (int64_t)(((uint64_t)(uint32_t)uni((int)(x >> 32)) << 32) | (uint32_t)uni((int)(uint32_t)x));
}

// Inclusive prefix sum across the wave.
__device__ __forceinline__ int64_t wave_incl_scan64(int64_t v, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int64_t t = __shfl_up(v, off, kWave);
    if (lane >= off) v += t;
  }
  return v;
}

// Operands of one 32-key chunk, loaded ahead of their use.
struct Chunk {
  u32x4 ka[4], kb[4], v[8];
  int kv0;
  bool vok;
};

// A workgroup holds four waves. Split (FULL): each wave walks a span of its
// own. Whole ranges (an SWA window, or a FULL context of one pass: only
// sequences x head groups items, each a short chain of dependent chunk
// loads): the four waves share one item, take every fourth chunk of its
// range, and combine their partial softmax states through LDS (still one
// pass: no workspace and no second kernel).
constexpr int kWaves = 4;
template <bool kSplit>
constexpr int kCoop = kSplit ? 1 : kWaves;  // waves that share one item

// kCGd: 16-column MFMA groups per wave. With two groups (several queries: 32
// (query, head) columns of a KV head) one wave scores both against the same
// K/V loads, which halves the KV bytes read. Whole-range items: with one group
// a wave has at most 168 VGPRs, so that three waves share a SIMD (two with two
// groups). Split spans with one page per chunk (PG >= 32): one wave per SIMD,
// which leaves room for two chunks of operands in flight.
template <bool kSplit, bool kOnePage, int kCGd>
__global__ __launch_bounds__(kWave * kWaves) __attribute__((amdgpu_waves_per_eu(kSplit && kOnePage ? 1 : (kCGd == 1 ? 3 : 2))))
void decode_kernel(DecodeParams p) {
  const PoolView &pv = p.pool;
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x >> 6;  // wave of the workgroup
  const int r = lane & 15, q = lane >> 4;
  const int hkv = p.hkv;
  const int shift = pv.pg_shift;
  const int pg = 1 << shift;
  const float c2 = p.scale_log2;
  const int ncols = p.nq * p.group;  // (query, head) pairs of one KV head
  const int hchunks = (ncols + kCols * kCGd - 1) / (kCols * kCGd);  // column items per KV head

  // Loop-invariant byte offsets of this lane's operands inside one 32-key K
  // block (used when a 32-key chunk never straddles two pages, i.e. PG >= 32):
  // slab t of half a (keys 8i + j, j < 4: MFMA rows 4i + j) is the A operand
  // of step t in lane order, a contiguous 1 KiB; half b (keys 8i + 4 + j) 4 KiB on.
  const uint32_t koff_a = lane * 16;
  const uint32_t koff_b = koff_a + 4096;
  // V^T of a 32-key chunk is one [D][32] block when PG >= 32: lane reads dims
  // 16 dt + r, keys 8 q .. 8 q + 7 of it.
  const uint32_t voff = (r * 32 + 8 * q) * 2;
  const uint32_t vstep = 16 * 32 * 2;  // 16 dims of a V block

  // Which work this wave runs. Whole ranges: one item per workgroup, in
  // (sequence, head group) order. Split (FULL layers): the 32-key chunks of
  // every (sequence, head group) segment, in (sequence, head group, chunk)
  // order, are cut into equal spans of `per` chunks, one span per wave of a
  // grid sized to the waves the device holds at once; a wave walks its span
  // across segment boundaries. A segment's pieces are its intersections with
  // the spans (piece k of a segment starting at unit S lies in span S / per + k),
  // which the merge kernel recomputes from the same lengths. The chunk cuts
  // are logical positions, so results do not depend on physical pages.
  const int H = hkv * hchunks;
  int b = 0, gy = 0;
  int64_t u = 0, u1 = 0, per = 1, pb = 0;  // span [u, u1) in units; pb: first unit of sequence b
  int nch = 0, c_lo = 0;                   // nch: chunks of sequence b
  if constexpr (kSplit) {
    const int64_t w = (int64_t)blockIdx.x * kWaves + wid;
    int64_t total = 0;
    for (int s0 = 0; s0 < p.ns; s0 += kWave) total += wave_sum64(seq_chunks(p, s0 + lane));
    total = uni64(total) * H;
    per = max((int64_t)(p.split_len / kChunk), (total + p.span_waves - 1) / p.span_waves);
    u = w * per;
    if (u >= total) return;
    u1 = min(total, u + per);
    int64_t base = 0;
    for (int b0 = 0;; b0 += kWave) {  // the sequence holding unit u (one exists: u < total)
      const int nchl = seq_chunks(p, b0 + lane);
      const int64_t incl = wave_incl_scan64((int64_t)H * nchl, lane);
      const int64_t tot = uni64(__shfl(incl, kWave - 1, kWave));
      if (u < base + tot) {
        const int first = __builtin_ctzll(__ballot(base + incl > u));
        b = b0 + first;
        nch = uni(__shfl(nchl, first, kWave));
        pb = base + uni64(__shfl(incl, first, kWave)) - (int64_t)H * nch;
        break;
      }
      base += tot;
    }
    gy = (int)((u - pb) / nch);
    c_lo = (int)(u - pb - (int64_t)gy * nch);
  } else {
    const int64_t item = blockIdx.x;
    if (item >= (int64_t)p.ns * H) return;
    b = (int)(item / H);
    gy = (int)(item % H);
  }
  for (;;) {
    // split: chunks [c_lo, c_hi) of segment (b, gy) are piece `piece` of it;
    // `whole` when they are all of it (the output row is then written here)
    int c_hi = 0, piece = 0;
    bool whole = true;
    if constexpr (kSplit) {
      const int64_t seg = pb + (int64_t)gy * nch;
      c_hi = (int)min((int64_t)nch, c_lo + (u1 - u));
      piece = (int)((seg + c_lo) / per - seg / per);
      whole = c_lo == 0 && c_hi == nch;
    }
    {
      const int g = gy / hchunks;
      const int hc = gy - g * hchunks;
      // this lane's MFMA column in group cg: query qi of the sequence, head hh of
      // KV head g's group
      int qi[kCGd];
      bool colv[kCGd];
      int64_t row[kCGd];  // output rows (where colv)
#pragma unroll
      for (int cg = 0; cg < kCGd; ++cg) {
        const int col = (hc * kCGd + cg) * kCols + r;
        colv[cg] = col < ncols;
        qi[cg] = colv[cg] ? col / p.group : 0;
        const int hh = colv[cg] ? col - qi[cg] * p.group : 0;
        row[cg] = ((int64_t)b * p.nq + qi[cg]) * p.hq + (int64_t)g * p.group + hh;
      }

      const int ctx = min(p.ctx_lens[b], p.max_ctx);
      if (ctx < 1) {
        if (!kSplit && wid == 0) {
          const u32x2 z = {0u, 0u};
#pragma unroll
          for (int cg = 0; cg < kCGd; ++cg)
            if (colv[cg]) {
#pragma unroll
              for (int dt = 0; dt < 8; ++dt)
                *reinterpret_cast<u32x2 *>(p.out + row[cg] * kHeadDim + 16 * dt + 4 * q) = z;
            }
        }
        return;
      }
      const int pos = ctx - 1;       // the last query's position
      const int pos0 = ctx - p.nq;   // the first query's position
      int kb, ke;                    // the item's key range (union over its columns)
      if (kSplit) {
        kb = c_lo * kChunk;
        ke = min(pos, c_hi * kChunk - 1);
      } else {
        kb = pv.window > 0 ? max(0, pos0 - pv.window + 1) : 0;
        ke = pos;
      }
      // keys this lane's columns may see: causal among the queries, and their window
      int ckb[kCGd], cke[kCGd];
#pragma unroll
      for (int cg = 0; cg < kCGd; ++cg) {
        const int cpos = pos0 + qi[cg];
        ckb[cg] = max(kb, pv.window > 0 ? max(0, cpos - pv.window + 1) : 0);
        cke[cg] = min(ke, cpos);
      }

      // Q^T operands: lane holds column r of group cg, dims 32t + 8q .. +7 for step t.
      u32x4 qf[kCGd][4];
#pragma unroll
      for (int cg = 0; cg < kCGd; ++cg) {
        const uint16_t *qrow = p.q + (colv[cg] ? row[cg] : (int64_t)b * p.nq * p.hq) * kHeadDim;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const u32x4 v = ldg128(qrow + 32 * t + 8 * q);
          const u32x4 z = {0u, 0u, 0u, 0u};
          qf[cg][t] = colv[cg] ? v : z;
        }
      }

      const int cfirst = kb & ~(kChunk - 1);
      const int nchunks = ((ke - cfirst) >> 5) + 1;
      const int c0 = kSplit ? 0 : wid;  // first chunk of this wave
      const int klo8 = kb & ~7, khi8 = ke & ~7;
      const int last_lp = ke >> shift;

      LaneTable tab;
      load_lane_table(tab, pv, b, kb >> shift, last_lp, lane);

      // Running column maxima in exp2 units (score * scale * log2 e): a finite
      // start whatever the scale, raised lazily (see scores).
      float m[kCGd], lsum[kCGd];
      f32x4 acc[kCGd][8];
#pragma unroll
      for (int cg = 0; cg < kCGd; ++cg) {
        m[cg] = -FLT_MAX;
        lsum[cg] = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[cg][i] = f32x4{0.f, 0.f, 0.f, 0.f};
      }

      auto issue_k = [&](int c, int page, Chunk &ch) {
        const int cbase = cfirst + c * kChunk;
        const int64_t pg64 = max(page, 0);
        const char *kbase = reinterpret_cast<const char *>(pv.k_pool) +
                            ((((pg64 * hkv + g) << shift) + (cbase & (pg - 1))) * kHeadDim) * 2;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          ch.ka[t] = ldnt128(kbase + koff_a + 1024 * t);
          ch.kb[t] = ldnt128(kbase + koff_b + 1024 * t);
        }
      };
      auto issue_v = [&](int c, int page, Chunk &ch) {
        const int cbase = cfirst + c * kChunk;
        const int64_t pg64 = max(page, 0);
        // PG >= 32 here, so VB = 32: the chunk is block (cbase mod PG) / 32 of the page-head
        const char *vbase = reinterpret_cast<const char *>(pv.v_pool) +
                            ((((pg64 * hkv + g) << shift) << kHeadDimShift) +
                             ((int64_t)((cbase & (pg - 1)) >> 5) << (5 + kHeadDimShift))) * 2;
        ch.kv0 = cbase + 8 * q;
        ch.vok = page >= 0;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) ch.v[dt] = ldnt128(vbase + voff + dt * vstep);
      };
      // General path (PG = 16: a chunk spans two pages): per-lane page choice.
      auto issue = [&](int c, Chunk &ch) {
        const int cbase = cfirst + c * kChunk;
        const int lpc = max(cbase, kb) >> shift;  // first page of the chunk's valid keys
        if ((min(cbase + kChunk - 1, ke) >> shift) - tab.lp0 >= kWave) load_lane_table(tab, pv, b, lpc, last_lp, lane);
        const int rel = lpc - tab.lp0;
        const int pg0 = __builtin_amdgcn_readlane(tab.page, rel);
        const int pg1 = __builtin_amdgcn_readlane(tab.page, min(rel + 1, kWave - 1));
        const int ka = min(max(cbase + 8 * (r >> 2) + (r & 3), kb), ke);
        const int kb2 = min(max(cbase + 8 * (r >> 2) + 4 + (r & 3), kb), ke);
        const int kvg = min(max(cbase + 8 * q, klo8), khi8);
        const int pa = (ka >> shift) == lpc ? pg0 : pg1;
        const int pb = (kb2 >> shift) == lpc ? pg0 : pg1;
        const int pvv = (kvg >> shift) == lpc ? pg0 : pg1;
        ch.kv0 = cbase + 8 * q;
        ch.vok = pvv >= 0;
        const int64_t pa64 = max(pa, 0), pb64 = max(pb, 0), pv64 = max(pvv, 0);
        // dims 32 t + 8 q .. +7 of a key: slab t of its half, 16 * B elements apart
        const int64_t kstep = (int64_t)16 << pv.vb_shift;
        const uint16_t *krow_a = pv.k_pool + k_offset(pv, pa64, hkv, g, ka & (pg - 1), 8 * q);
        const uint16_t *krow_b = pv.k_pool + k_offset(pv, pb64, hkv, g, kb2 & (pg - 1), 8 * q);
        const uint16_t *vcol = pv.v_pool + v_offset(pv, pv64, hkv, g, kvg & (pg - 1), r);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          ch.ka[t] = ldnt128(krow_a + kstep * t);
          ch.kb[t] = ldnt128(krow_b + kstep * t);
        }
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) ch.v[dt] = ldnt128(vcol + ((int64_t)(16 * dt) << pv.vb_shift));
      };

      // QK^T and the online softmax of one chunk: returns P^T packed as bf16 and
      // leaves the key mask in `keep`. The running maximum of a column is only
      // raised when one of its scores exceeds it by more than 2^8 in exp2 units
      // (a ballot over the lanes' own maxima; the exact column maximum is formed
      // only then), so the output rescale is rare; numerator and denominator
      // share the stale maximum, so the result is exact. Starting from -FLT_MAX
      // (exp2 units), a masked score (-inf) gives probability 0 without
      // (-inf) - (-inf), and the first finite score always raises the maximum
      // (alpha = 0).
      uint32_t keep = 0;
      auto qk = [&](const Chunk &ch, f32x4 (&sa)[kCGd], f32x4 (&sb)[kCGd]) {
#pragma unroll
        for (int cg = 0; cg < kCGd; ++cg) sa[cg] = sb[cg] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int cg = 0; cg < kCGd; ++cg) {
            sa[cg] = mfma16x16x32(ch.ka[t], qf[cg][t], sa[cg]);
            sb[cg] = mfma16x16x32(ch.kb[t], qf[cg][t], sb[cg]);
          }
      };
      auto softmax = [&](const Chunk &ch, const f32x4 (&sa)[kCGd], const f32x4 (&sb)[kCGd], u32x4 (&pf)[kCGd]) {
        // keep: keys of the item range (V rows outside it are zeroed below);
        // sk: those this lane's column sees. Interior chunks have all bits set
        // and skip the per-score masking (a wave-uniform branch).
        keep = ch.vok ? key_bits(ch.kv0, kb, ke) : 0u;
#pragma unroll
        for (int cg = 0; cg < kCGd; ++cg) {
          const uint32_t sk = keep & key_bits(ch.kv0, ckb[cg], cke[cg]);
          float s[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            s[i] = sa[cg][i];
            s[4 + i] = sb[cg][i];
          }
          if (__builtin_amdgcn_ballot_w64(sk != 0xFFu) != 0) {
#pragma unroll
            for (int i = 0; i < 8; ++i) s[i] = (sk >> i) & 1u ? s[i] : -INFINITY;
          }
          const float lmax = max8(s) * c2;
          if (__builtin_amdgcn_ballot_w64(lmax > m[cg] + kRescaleLog2) != 0) {
            const float cmax = max_xor32(max_xor16(lmax));
            const bool up = cmax > m[cg] + kRescaleLog2;
            const float alpha = up ? fast_exp2(m[cg] - cmax) : 1.f;
            m[cg] = up ? cmax : m[cg];
            lsum[cg] *= alpha;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) acc[cg][dt] *= alpha;
          }
          const float mc = m[cg];
          float pr[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) pr[i] = fast_exp2(fmaf(s[i], c2, -mc));
#pragma unroll
          for (int j = 0; j < 4; ++j) pf[cg][j] = pack_bf16x2(pr[2 * j], pr[2 * j + 1]);
#pragma unroll
          for (int j = 0; j < 4; ++j) lsum[cg] = dot2_bf16_ones(pf[cg][j], lsum[cg]);
        }
      };
      auto scores = [&](Chunk &ch, u32x4 (&pf)[kCGd]) {
        f32x4 sa[kCGd], sb[kCGd];
        qk(ch, sa, sb);
        softmax(ch, sa, sb, pf);
      };
      auto pv_update = [&](Chunk &ch, const u32x4 (&pf)[kCGd]) {
        if (keep != 0xFFu) {
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) ch.v[dt] = keep_bf16x8(ch.v[dt], keep);
        }
#pragma unroll
        for (int dt = 0; dt < 8; ++dt)
#pragma unroll
          for (int cg = 0; cg < kCGd; ++cg) acc[cg][dt] = mfma16x16x32(ch.v[dt], pf[cg], acc[cg][dt]);
      };

      // One-page path (PG >= 32): a chunk's keys lie in one page.
      if constexpr (kOnePage) {
        // chunks come in increasing order: the lane table moves forward when a
        // chunk's page lies past its 64 entries
        auto page_of = [&](int c) {
          const int lp = (cfirst + c * kChunk) >> shift;
          if (lp - tab.lp0 >= kWave) load_lane_table(tab, pv, b, lp, last_lp, lane);
          return __builtin_amdgcn_readlane(tab.page, lp - tab.lp0);
        };
        // this wave's chunks: c0, c0 + kCoop, ...
        const int nw = nchunks > c0 ? (nchunks - c0 + kCoop<kSplit> - 1) / kCoop<kSplit> : 0;
        // Fused append (split spans, one query per sequence): the piece that
        // holds the segment's last chunk holds the step's token at `pos`. Its
        // key is not in the pool yet: this lane's pieces of it come from
        // k_new / v_new and replace what the chunk's loads read for that key,
        // and the first head group's wave stores the row in its slot.
        const bool app = kSplit && p.split_append && nw > 0 && c_hi == nch;
        u32x4 kapp[4];
        uint32_t vapp[8];
        int app_page = -1;  // the token's page (-1: invalid, nothing stored)
        if (app) {
          const int64_t kvrow = ((int64_t)b * hkv + g) * kHeadDim;
#pragma unroll
          for (int t = 0; t < 4; ++t) kapp[t] = ldg128(p.k_new + kvrow + 32 * t + 8 * q);
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) vapp[dt] = p.v_new[kvrow + 16 * dt + r];
          const int lp = pos >> shift;
          if (lp < pv.stride) {
            const int64_t v = pv.table[(int64_t)b * pv.stride + lp];
            app_page = v >= 0 && v < pv.num_pages ? (int)v : -1;
          }
        }
        // the new key kc = pos % 32 of the last chunk: K rows of MFMA row
        // 4 (kc / 8) + kc % 4 in half (kc / 4) % 2 (dims 32 t + 8 q .. +7 in
        // lane r + 16 q); V pieces of lanes q = kc / 8, element kc % 8
        auto patch = [&](Chunk &ch) {
          const int kc = pos & (kChunk - 1);
          const bool kl = r == 4 * (kc >> 3) + (kc & 3);
          const bool hb = (kc >> 2) & 1;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            ch.ka[t] = kl && !hb ? kapp[t] : ch.ka[t];
            ch.kb[t] = kl && hb ? kapp[t] : ch.kb[t];
          }
          const bool vl = q == (kc >> 3);
          const int e = kc & 7, sh = 16 * (e & 1);
          const uint32_t msk = 0xFFFFu << sh;
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const uint32_t w = (ch.v[dt][j] & ~msk) | (vapp[dt] << sh);
              ch.v[dt][j] = vl && j == (e >> 1) ? w : ch.v[dt][j];
            }
          }
        };
        if (kSplit && nw > 0) {
          // Split spans (long streams of chunks): one wave per SIMD, two whole
          // chunks in flight while a third is computed. Chunk k is computed
          // while k + 1 is loaded and k + 2 is issued right after k's products;
          // past the span's end the last chunk is loaded again (never used),
          // so that every wait counts the same loads.
          Chunk ca, cb;
          auto issue_both = [&](int k, Chunk &ch) {
            const int cc = c0 + k * kCoop<kSplit>;
            const int page = page_of(cc);
            issue_k(cc, page, ch);
            issue_v(cc, page, ch);
          };
          issue_both(0, ca);
          issue_both(min(1, nw - 1), cb);
          if (app && hc == 0 && app_page >= 0) {
            // the append, early so that its stores are done long before the
            // kernel ends: the token's K row (lanes r = 0 hold dims
            // 32 t + 8 q) and V column (lanes q = 0 hold dims 16 dt + r)
            const int o = pos & (pg - 1);
            if (r == 0) {
#pragma unroll
              for (int t = 0; t < 4; ++t)
                stg128(pv.k_pool + k_offset(pv, app_page, hkv, g, o, 32 * t + 8 * q), kapp[t]);
            }
            if (q == 0) {
#pragma unroll
              for (int dt = 0; dt < 8; ++dt) pv.v_pool[v_offset(pv, app_page, hkv, g, o, 16 * dt + r)] = (uint16_t)vapp[dt];
            }
          }
          u32x4 pf[kCGd];
          int k = 0;
          // the last chunk (index nw - 1) is the loop's second one or the tail's
          for (; k + 2 <= nw; k += 2) {
            scores(ca, pf);
            pv_update(ca, pf);
            __builtin_amdgcn_sched_barrier(0);
            issue_both(min(k + 2, nw - 1), ca);
            __builtin_amdgcn_sched_barrier(0);
            if (app && k + 1 == nw - 1) patch(cb);
            scores(cb, pf);
            pv_update(cb, pf);
            __builtin_amdgcn_sched_barrier(0);
            issue_both(min(k + 3, nw - 1), cb);
            __builtin_amdgcn_sched_barrier(0);
          }
          if (k < nw) {
            if (app) patch(ca);
            scores(ca, pf);
            pv_update(ca, pf);
          }
        } else if (nw > 0) {
          Chunk ch;
          {
            const int page = page_of(c0);
            issue_k(c0, page, ch);
            issue_v(c0, page, ch);
          }
          // The scheduling fences keep each chunk's loads behind the last use of
          // the registers they overwrite: one operand set, no loop-carried copies.
          // The next K loads go out as soon as QK^T has read this chunk's K, ahead
          // of the softmax, so that a full chunk of loads stays in flight.
          u32x4 pf[kCGd];
          for (int k = 0; k < nw - 1; ++k) {
            const int cn = c0 + (k + 1) * kCoop<kSplit>;
            const int next_page = page_of(cn);
            f32x4 sa[kCGd], sb[kCGd];
            qk(ch, sa, sb);
            __builtin_amdgcn_sched_barrier(0);
            issue_k(cn, next_page, ch);
            __builtin_amdgcn_sched_barrier(0);
            softmax(ch, sa, sb, pf);
            pv_update(ch, pf);
            __builtin_amdgcn_sched_barrier(0);
            issue_v(cn, next_page, ch);
            __builtin_amdgcn_sched_barrier(0);
          }
          scores(ch, pf);
          pv_update(ch, pf);
        }
      } else {
        for (int c = c0; c < nchunks; c += kCoop<kSplit>) {
          Chunk ch;
          u32x4 pf[kCGd];
          issue(c, ch);
          scores(ch, pf);
          pv_update(ch, pf);
        }
      }

      // Lane holds O^T[d = 16 dt + 4 q + i][column r of group cg], relative to
      // its column maximum m.
      if constexpr (!kSplit) {
        // Combine the kCoop waves' partial states through LDS; wave w then
        // normalises and writes dims 32 w .. 32 w + 31 of every column.
        // s_o keeps each lane's accumulator vectors in lane order (16-B stores and
        // loads, no bank conflicts)
        __shared__ f32x4 s_o[kCoop<kSplit>][kCGd][8][kWave];
        __shared__ float s_m[kCoop<kSplit>][kCGd][kCols], s_l[kCoop<kSplit>][kCGd][kCols];
#pragma unroll
        for (int cg = 0; cg < kCGd; ++cg) {
          const float l = sum_xor32(sum_xor16(lsum[cg]));
          if (q == 0) {
            s_m[wid][cg][r] = m[cg];
            s_l[wid][cg][r] = l;
          }
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) s_o[wid][cg][dt][lane] = acc[cg][dt];
        }
        __syncthreads();
        // this lane's 8 output dims d0 .. d0 + 7: dims 16 dt + 4 q' + i of the
        // accumulators with dt = 2 wid + q / 2 and q' = 2 (q % 2), 2 (q % 2) + 1
        const int d0 = 32 * wid + 8 * q;
        const int sdt = 2 * wid + (q >> 1), sl = r + 32 * (q & 1);
#pragma unroll
        for (int cg = 0; cg < kCGd; ++cg) {
          if (!colv[cg]) continue;
          float mx = -FLT_MAX;
#pragma unroll
          for (int w = 0; w < kCoop<kSplit>; ++w) mx = fmaxf(mx, s_m[w][cg][r]);
          float wgt[kCoop<kSplit>], l = 0.f;
#pragma unroll
          for (int w = 0; w < kCoop<kSplit>; ++w) {
            wgt[w] = fast_exp2(s_m[w][cg][r] - mx);
            l += wgt[w] * s_l[w][cg][r];
          }
          // a column that sees no key at all (a query before position 0) writes zeros
          const float inv = l > 0.f ? 1.f / l : 0.f;
          f32x4 o0 = {0.f, 0.f, 0.f, 0.f}, o1 = o0;
#pragma unroll
          for (int w = 0; w < kCoop<kSplit>; ++w) {
            o0 += wgt[w] * s_o[w][cg][sdt][sl];
            o1 += wgt[w] * s_o[w][cg][sdt][sl + 16];
          }
          const float o[8] = {o0[0] * inv, o0[1] * inv, o0[2] * inv, o0[3] * inv,
                              o1[0] * inv, o1[1] * inv, o1[2] * inv, o1[3] * inv};
          u32x4 wv;
#pragma unroll
          for (int j = 0; j < 4; ++j) wv[j] = pack_bf16x2(o[2 * j], o[2 * j + 1]);
          *reinterpret_cast<u32x4 *>(p.out + row[cg] * kHeadDim + d0) = wv;
        }
      } else {
#pragma unroll
        for (int cg = 0; cg < kCGd; ++cg) {
          const float l = sum_xor32(sum_xor16(lsum[cg]));
          if (!colv[cg]) continue;
          // a column that sees no key of this piece (a later query's last keys)
          // writes o = 0 with log-sum-exp -inf: weight 0 in the merge
          const float inv = l > 0.f ? 1.f / l : 0.f;
          if (whole) {  // the only piece: the normalised row (zeros if it sees no key)
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
              const f32x4 o = acc[cg][dt] * inv;
              u32x2 wv;
              wv[0] = pack_bf16x2(o[0], o[1]);
              wv[1] = pack_bf16x2(o[2], o[3]);
              *reinterpret_cast<u32x2 *>(p.out + row[cg] * kHeadDim + 16 * dt + 4 * q) = wv;
            }
            continue;
          }
          float *dst = p.ws_o + (row[cg] * p.max_splits + piece) * kHeadDim + 4 * q;
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) *reinterpret_cast<f32x4 *>(dst + 16 * dt) = acc[cg][dt] * inv;
          if (q == 0) p.ws_lse[row[cg] * p.max_splits + piece] = m[cg] + __log2f(l);
        }
      }
    }
    if constexpr (!kSplit) {
      break;
    } else {
      // next segment of the span: the next head group, else the next sequence
      // with keys (one exists while u < u1)
      u += c_hi - c_lo;
      if (u >= u1) break;
      c_lo = 0;
      if (++gy == H) {
        gy = 0;
        pb += (int64_t)H * nch;
        do nch = uni(seq_chunks(p, ++b));  // a scalar load
        while (nch == 0);
      }
    }
  }
}

// Log-sum-exp merge of the split partials: one wave per (sequence, query, head).
// Lane j reads the log-sum-exp of pieces j, j+64, ...; the weights are then
// broadcast by readlane while the two half-waves accumulate even and odd
// pieces, four output dims a lane (16-byte loads, 16 pieces in flight a step).
__global__ __launch_bounds__(kMergeThreads) void decode_merge_kernel(DecodeParams p) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t idx = (int64_t)blockIdx.x * (kMergeThreads / kWave) + (threadIdx.x / kWave);
  if (idx >= (int64_t)p.ns * p.nq * p.hq) return;
  const int b = (int)(idx / ((int64_t)p.nq * p.hq));
  const int ctx = min(p.ctx_lens[b], p.max_ctx);
  const int half = lane >> 5, d4 = (lane & 31) * 4;
  u32x2 *dst = reinterpret_cast<u32x2 *>(p.out + idx * kHeadDim + d4);
  const u32x2 zero = {0u, 0u};
  if (ctx < 1) {
    if (half == 0) *dst = zero;
    return;
  }
  // the row's segment and the spans of the decode grid (same arithmetic as there)
  const int hchunks = (p.nq * p.group + p.item_cols - 1) / p.item_cols;
  const int H = p.hkv * hchunks;
  int64_t total = 0, pb = 0;
  for (int s0 = 0; s0 < p.ns; s0 += kWave) {
    const int n = seq_chunks(p, s0 + lane);
    total += wave_sum64(n);
    pb += wave_sum64(s0 + lane < b ? n : 0);
  }
  total = uni64(total) * H;
  pb = uni64(pb) * H;
  const int64_t per = max((int64_t)(p.split_len / kChunk), (total + p.span_waves - 1) / p.span_waves);
  const int rem = (int)(idx - (int64_t)b * p.nq * p.hq);
  const int qi = rem / p.hq, head = rem - qi * p.hq;
  const int g = head / p.group;
  const int col = qi * p.group + (head - g * p.group);
  const int nch = (ctx + kChunk - 1) / kChunk;
  const int64_t seg = pb + (int64_t)(g * hchunks + col / p.item_cols) * nch;
  const int nsplit = (int)((seg + nch - 1) / per - seg / per) + 1;
  if (nsplit == 1) return;  // one piece: the decode kernel wrote the row
  const float *lse = p.ws_lse + idx * p.max_splits;
  float mx = -INFINITY;
  for (int s = lane; s < nsplit; s += kWave) mx = fmaxf(mx, lse[s]);
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
  mx = max_xor32(max_xor16(mx));
  if (mx == -INFINITY) {  // a query that sees no key (multi-query rows before position 0)
    if (half == 0) *dst = zero;
    return;
  }
  const float *po = p.ws_o + idx * p.max_splits * kHeadDim + d4;
  float wsum = 0.f;
  f32x4 o = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < nsplit; s0 += kWave) {
    const int s = s0 + lane;
    const float w = s < nsplit ? fast_exp2(lse[s] - mx) : 0.f;
    const int n = min(kWave, nsplit - s0);
    for (int k0 = 0; k0 < n; k0 += 16) {
      f32x4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int pc = k0 + 2 * k + half;
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        v[k] = pc < n ? *reinterpret_cast<const f32x4 *>(po + (int64_t)(s0 + pc) * kHeadDim) : z;
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int pe = min(k0 + 2 * k, kWave - 1), pd = min(k0 + 2 * k + 1, kWave - 1);
        const float we = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), pe));
        const float wd = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), pd));
        const int pc = k0 + 2 * k + half;
        const float wk = pc < n ? (half ? wd : we) : 0.f;
        wsum += wk;
        o += wk * v[k];
      }
    }
  }
  // the two halves hold even and odd pieces: add across lanes l and l ^ 32
  wsum = sum_xor32(wsum);
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = sum_xor32(o[i]);
  const float inv = 1.f / wsum;
  if (half == 0) {
    u32x2 w2;
    w2[0] = pack_bf16x2(o[0] * inv, o[1] * inv);
    w2[1] = pack_bf16x2(o[2] * inv, o[3] * inv);
    *dst = w2;
  }
}

}  // namespace

int32_t decode_split_len(int32_t ns, int32_t hkv, int32_t group, int32_t max_ctx) {
  // The fewest keys of a wave's span: 256 to 2048, larger for larger batches
  // (about 8192 spans of this length when contexts average half the maximum),
  // so that spans of small batches stay short enough to fill the device and
  // the workspace stays bounded; very long contexts get longer spans so that a
  // row has at most 257 pieces.
  const int64_t heads = (int64_t)hkv * ((group + kCols - 1) / kCols);
  const int64_t keys = heads * ns * (int64_t)max_ctx / 2;
  int32_t len = 256;
  while (len < 2048 && keys / (2 * len) >= 8192) len *= 2;
  const int64_t min_len = ((int64_t)max_ctx + 255) / 256;
  while (len < min_len) len *= 2;
  return len;
}

// Waves of `kernel` the current device holds at once (workgroups per CU from
// its register and LDS use, times the CUs), looked up once per device.
template <bool kOnePage, int kCGd>
hipError_t resident_split_waves(int &waves) {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cache[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < kMaxDevices && (waves = cache[dev].load(std::memory_order_relaxed)) > 0) return hipSuccess;
  int cus = 0, blocks = 0;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_kernel<true, kOnePage, kCGd>, kWave * kWaves,
                                                        0)) != hipSuccess)
    return e;
  waves = max(1, cus) * max(1, blocks) * kWaves;
  if (dev >= 0 && dev < kMaxDevices) cache[dev].store(waves, std::memory_order_relaxed);
  return hipSuccess;
}

template <int kCGd>
hipError_t launch_decode_cg(const DecodeParams &p0, hipStream_t stream) {
  DecodeParams p = p0;
  p.item_cols = kCols * kCGd;
  const int hitems = (p.nq * p.group + p.item_cols - 1) / p.item_cols;
  const int64_t items = (int64_t)p.ns * p.hkv * hitems;  // whole range: one item per workgroup
  // One-page path: 32-key chunks never straddle pages (PG >= 32).
  const bool one_page = p.pool.pg_shift >= 5;
  const dim3 block(kWave * kWaves);
  if (p.max_splits > 1) {
    hipError_t e = one_page ? resident_split_waves<true, kCGd>(p.span_waves)
                            : resident_split_waves<false, kCGd>(p.span_waves);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(p.span_waves / kWaves));
    e = one_page ? launch_kernel(decode_kernel<true, true, kCGd>, grid, block, stream, p)
                 : launch_kernel(decode_kernel<true, false, kCGd>, grid, block, stream, p);
    if (e != hipSuccess) return e;
    const int64_t rows = (int64_t)p.ns * p.nq * p.hq;
    const int per_block = kMergeThreads / kWave;
    return launch_kernel(decode_merge_kernel, dim3((unsigned)((rows + per_block - 1) / per_block)),
                         dim3(kMergeThreads), stream, p);
  }
  return one_page ? launch_kernel(decode_kernel<false, true, kCGd>, dim3((unsigned)items), block, stream, p)
                  : launch_kernel(decode_kernel<false, false, kCGd>, dim3((unsigned)items), block, stream, p);
}

hipError_t launch_decode(const DecodeParams &p, hipStream_t stream) {
  if (p.ns <= 0) return hipSuccess;
  // more than 16 (query, head) columns per KV head: one wave takes 32 of them
  return p.nq * p.group > kCols ? launch_decode_cg<2>(p, stream) : launch_decode_cg<1>(p, stream);
}

}  // namespace hswa
