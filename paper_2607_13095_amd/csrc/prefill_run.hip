// Windowed (SWA) chunked prefill, persistent over runs of position tiles.
//
// "Compute Analysis": an SWA layer's attention covers a local window, so its
// prefill is bound by moving q, o and the chunk's K/V rather than by the
// matrix cores. A workgroup that serves one tile of positions has to stage the
// whole window (W + positions - 1 keys) for that tile alone, so every key is
// staged about W / positions times. Here one workgroup (16 waves of 16 rows)
// walks a run of consecutive tiles of one (sequence, KV head) pair instead:
// tile t holds 256 query rows (a row = a (position, query head) pair of the KV
// head's GQA group, so 256 / G positions), the window's 32-key chunks stay in
// an LDS ring of eight, and each tile stages only the chunk its last positions
// add. The chunk a tile will need next is loaded into registers while the tile
// computes (waves 0-7 carry its V, waves 8-15 its K); each wave loads its
// next tile's queries as soon as its last QK^T of the tile has read the
// current ones; waves run through a tile's chunks without barriers (one
// barrier per tile). Tiles whose positions all exist issue their loads and
// stores unconditionally, so the memory counters stay exact along the loop
// and no wait covers more than the operation it is for.
//
// Used when G >= 8 and W + 256 / G - 1 <= 160: a tile then spans at most 7
// chunks and the next tile adds at most one, so the ring of 8 is never short.
// Per 32-key chunk and wave (bf16 MFMA, fp32 accumulate), as in the other
// prefill kernels:
//   S^T[key][row] = K[key][:] . Q[row][:]     (Q held in registers)
//   online softmax per row (exp2, scale * log2 e folded in, running maximum in
//   exp2 units, raised lazily)
//   O^T[d][row]  += V^T[d][key] . P^T[key][row]
// LDS holds each chunk in MFMA operand order (K: the pool's K block layout;
// V^T: block dt for lane r + 16 q = keys 8 q .. +7 of dim 16 dt + r). Cached
// keys are chunked at 32-aligned positions and the chunk's own keys from P
// on, so no chunk mixes the two sources; keys outside the run's range are
// staged as zeros and every column masks its own window.
#include <algorithm>
#include <cfloat>
#include <type_traits>

#include "hswa_common.h"
#include "hswa_launch.h"

namespace hswa {
namespace {

constexpr int kRThreads = 1024;
constexpr int kRRows = 256;                      // query rows per tile (16 waves x 16)
constexpr int kRChunk = 32;                      // keys per chunk
constexpr int kRBufs = 8;                        // LDS ring of chunks
constexpr int kRKBytes = kRChunk * kHeadDim * 2; // 8 KiB of K per chunk
constexpr int kRBufBytes = 2 * kRKBytes;         // K, then V^T
constexpr int kRCG = 1;                          // 16-column MFMA groups per wave
constexpr float kRLaneSumLimit = 4096.f;         // lane share of a row sum that raises the maximum
constexpr int kRTargetGroups = 256;              // workgroups a launch aims for (one per CU)

// Staging registers of one chunk: waves 0-7 carry its V, waves 8-15 its K,
// one 16-byte piece a thread.
struct RStage {
  u32x4 a;
  uint32_t keep;  // K: bit 0 = the piece holds data; V: bits 0 .. 7 = its keys that do
};

__global__ __launch_bounds__(kRThreads) __attribute__((amdgpu_waves_per_eu(4))) void prefill_run_kernel(
    PrefillParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char s_lds[kRBufs * kRBufBytes];

  const PoolView &pv = p.pool;
  const int G = p.group;
  const int npos = kRRows / G;  // positions per tile
  const int ntq = (p.max_chunk_len + npos - 1) / npos;
  const int npairs = p.ns * p.hkv;
  const int runs = (int)(gridDim.x / npairs);
  const int tpr = (ntq + runs - 1) / runs;  // tiles per run
  const int pair = (int)(blockIdx.x / runs), run = (int)(blockIdx.x % runs);
  if (pair >= npairs) return;
  const int b = pair / p.hkv, g = pair - b * p.hkv;

  const int tok0 = p.cu_seqlens[b];
  const int C = min(min(p.cu_seqlens[b + 1], p.total_tokens) - tok0, p.max_chunk_len);
  const int P = p.prefix_lens[b];
  const int t0 = run * tpr;
  const int t1 = min((C + npos - 1) / npos, t0 + tpr);
  if (t0 >= t1 || P < 0 || tok0 < 0) return;
  const int W = pv.window;
  // keys of the whole run, cut at P into cached chunks (32-aligned) and new ones (aligned to P)
  const int klo = max(0, P + t0 * npos - W + 1);
  const int khi = P + min(C, t1 * npos) - 1;
  const int chi = min(P - 1, khi);  // last cached key (< klo: none)
  const int ncached = klo <= chi ? (chi >> 5) - (klo >> 5) + 1 : 0;
  const int nbase = max(klo, P) - P;
  const int nnew = khi >= max(klo, P) ? ((khi - P) >> 5) - (nbase >> 5) + 1 : 0;
  const int nch = ncached + nnew;
  auto chunk_base = [&](int c) {
    return c < ncached ? (klo & ~(kRChunk - 1)) + kRChunk * c : P + kRChunk * ((nbase >> 5) + c - ncached);
  };
  auto chunk_of = [&](int key) {
    return key < P ? (key >> 5) - (klo >> 5) : ncached + ((key - P) >> 5) - (nbase >> 5);
  };

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r = lane & 15, q = lane >> 4;
  const int hkv = p.hkv, hq = p.hq;
  const int shift = pv.pg_shift, pg = 1 << shift;
  const float c2 = p.scale_log2;

  // Page ids of the run's cached keys (at most W - 1 <= 159 keys, 12 pages of
  // 16): lane i holds the physical page of logical page lp0 + i, -1 if not
  // cached or not a valid page.
  const int lp0 = (klo & ~(kRChunk - 1)) >> shift;
  int tab = -1;
  if (ncached > 0) {
    const int lp = lp0 + lane;
    if (lp <= (chi >> shift)) {
      const int e = pv.ring > 0 ? lp % pv.ring : lp;
      if (e < pv.stride) {
        const int64_t v = pv.table[(int64_t)b * pv.stride + e];
        tab = (v >= 0 && v < pv.num_pages) ? (int)v : -1;
      }
    }
  }
  auto page_at = [&](int j) { return __shfl(tab, (j >> shift) - lp0, kWave); };

  // ---- staging ----
  // K piece idx (0 .. 511) of a chunk: dims 32 t + 8 qq .. +7 (t = (idx >> 6) & 3,
  // qq = (idx >> 4) & 3) of chunk key 8 ((idx & 15) >> 2) + 4 (idx >> 8) + (idx & 3),
  // at byte 16 idx of the K block. V^T piece idx: keys 8 qq .. +7 of dim
  // 16 (idx >> 6) + (idx & 15), at byte 16 idx of the V^T block.
  auto k_key = [](int idx) { return ((idx & 15) >> 2) * 8 + (idx >> 8) * 4 + (idx & 3); };
  auto k_dim = [](int idx) { return ((idx >> 6) & 3) * 32 + ((idx >> 4) & 3) * 8; };
  auto v_dim = [](int idx) { return (idx >> 6) * 16 + (idx & 15); };
  auto v_keys = [](int idx) { return ((idx >> 4) & 3) * 8; };
  const u32x4 zero = {0u, 0u, 0u, 0u};
  const bool vwave = wave < 8;   // waves 0-7 stage V, waves 8-15 stage K
  const int sidx = tid & 511;    // the piece this thread stages
  auto fetch = [&](int c, RStage &st) {
    c = min(c, nch - 1);  // past the end: a repeat of the last chunk, never stored
    const int kb = chunk_base(c);
    const bool cached = c < ncached;
    const uint16_t *src;
    uint32_t keep;
    if (vwave) {
      if (cached) {
        const int j0 = kb + v_keys(sidx);
        const int page = page_at(j0);
        src = pv.v_pool + v_offset(pv, page >= 0 ? page : 0, hkv, g, j0 & (pg - 1), v_dim(sidx));
        keep = page >= 0 ? key_range_bits(j0, klo, chi) : 0u;
      } else {
        // a row piece: key 4 wave + lane / 16, dims 8 (lane % 16) .. +7
        const int jv = kb + 4 * wave + (lane >> 4);
        const bool in = jv >= klo && jv <= khi;
        src = p.v_new + ((int64_t)(tok0 + (in ? jv - P : 0)) * hkv + g) * kHeadDim + (lane & 15) * 8;
        keep = in ? 0xFFu : 0u;
      }
    } else {
      const int j = kb + k_key(sidx);
      if (cached) {
        const int page = page_at(j);
        const bool in = j >= klo && j <= chi && page >= 0;
        src = pv.k_pool + k_offset(pv, in ? page : 0, hkv, g, j & (pg - 1), k_dim(sidx));
        keep = in ? 1u : 0u;
      } else {
        const bool in = j >= klo && j <= khi;
        src = p.k_new + ((int64_t)(tok0 + (in ? j - P : 0)) * hkv + g) * kHeadDim + k_dim(sidx);
        keep = in ? 1u : 0u;
      }
    }
    st.a = ldg128_global(src);
    st.keep = keep;
  };
  auto lds128 = [&](uint32_t off) { return reinterpret_cast<u32x4 *>(s_lds + off); };
  auto buf_off = [&](int buf) { return (uint32_t)__builtin_amdgcn_readfirstlane(buf * kRBufBytes); };
  // V^T byte of dim d = 8 (lane % 16) + 2 (lane / 16), keys 4 wave .. +3: the
  // 16-byte piece of key group wave / 2, its half wave % 2
  const int vd = 8 * (lane & 15) + 2 * (lane >> 4);
  const uint32_t st_vrow = kRKBytes + (((vd >> 4) * 64 + (vd & 15) + 16 * (wave >> 1)) * 16) + 8 * (wave & 1);
  // 4 x 4 transpose of dwords across the lanes l, l ^ 16, l ^ 32, l ^ 48.
  auto transpose4 = [&](const u32x4 &t, uint32_t (&w)[4]) {
    const auto a = __builtin_amdgcn_permlane32_swap(t[0], t[2], false, false);
    const auto bb = __builtin_amdgcn_permlane32_swap(t[1], t[3], false, false);
    const auto cc = __builtin_amdgcn_permlane16_swap((uint32_t)a[0], (uint32_t)bb[0], false, false);
    const auto d = __builtin_amdgcn_permlane16_swap((uint32_t)a[1], (uint32_t)bb[1], false, false);
    w[0] = (uint32_t)cc[0];
    w[1] = (uint32_t)cc[1];
    w[2] = (uint32_t)d[0];
    w[3] = (uint32_t)d[1];
  };
  auto store = [&](int c, const RStage &st) {
    const bool cached = c < ncached;
    const uint32_t bo = buf_off(c % kRBufs);
    if (!vwave) {
      *lds128(bo + 16 * sidx) = st.keep & 1u ? st.a : zero;
    } else if (cached) {
      const uint32_t k8 = st.keep & 0xFFu;
      *lds128(bo + kRKBytes + 16 * sidx) = k8 != 0xFFu ? keep_bf16x8(st.a, k8) : st.a;
    } else {
      // lanes l % 16 + 16 m hold key 4 wave + m x dims 8 (l % 16) .. +7; after
      // the transpose lane m holds dims 2 m, 2 m + 1 of keys 4 wave .. +3,
      // packed into half a V^T piece per dim
      uint32_t w[4];
      transpose4(st.keep & 1u ? st.a : zero, w);
      u32x2 lo, hi;
      lo[0] = __builtin_amdgcn_perm(w[1], w[0], 0x05040100u);
      lo[1] = __builtin_amdgcn_perm(w[3], w[2], 0x05040100u);
      hi[0] = __builtin_amdgcn_perm(w[1], w[0], 0x07060302u);
      hi[1] = __builtin_amdgcn_perm(w[3], w[2], 0x07060302u);
      *reinterpret_cast<u32x2 *>(s_lds + bo + st_vrow) = lo;
      *reinterpret_cast<u32x2 *>(s_lds + bo + st_vrow + 16) = hi;
    }
  };

  // ---- per-tile state ----
  u32x4 qf[kRCG][4];
  int cpos[kRCG], clo[kRCG];
  bool cval[kRCG];
  float m[kRCG], lsum[kRCG];  // m: running maximum in exp2 units
  f32x4 acc[kRCG][8];
  auto load_q = [&](int t) {
    const int q0 = t * npos, q1 = min(C, q0 + npos) - 1;
#pragma unroll
    for (int cg = 0; cg < kRCG; ++cg) {
      const int row = wave * (16 * kRCG) + cg * 16 + r;
      const int po = row / G, head = row - po * G;
      const bool ok = q0 + po <= q1;
      const int64_t tok = tok0 + q0 + (ok ? po : 0);
      const uint16_t *qrow = p.q + (tok * hq + (int64_t)g * G + head) * kHeadDim;
#pragma unroll
      for (int t4 = 0; t4 < 4; ++t4) qf[cg][t4] = ldg128(qrow + 32 * t4 + 8 * q);
    }
  };

  const uint32_t op_lane = lane * 16;
  // One chunk: QK^T, masks, online softmax (lazy maximum, exact), PV. With
  // `prefetch`, the next tile's queries are loaded right after the QK^T.
  // `first`: the wave's first chunk of the tile; its maximum is formed exactly
  // at once (the lazy check would always fail on it).
  auto chunk = [&](int c, int kb, int kend, int wint_lo, int wint_hi, bool first, bool prefetch, int tnext) {
    const uint32_t a = buf_off(c % kRBufs) + op_lane;
    f32x4 sc[2][kRCG];
#pragma unroll
    for (int ab = 0; ab < 2; ++ab)
#pragma unroll
      for (int cg = 0; cg < kRCG; ++cg) sc[ab][cg] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 ka = *lds128(a + 1024 * t);
      const u32x4 kbv = *lds128(a + 4096 + 1024 * t);
#pragma unroll
      for (int cg = 0; cg < kRCG; ++cg) {
        sc[0][cg] = mfma16x16x32(ka, qf[cg][t], sc[0][cg]);
        sc[1][cg] = mfma16x16x32(kbv, qf[cg][t], sc[1][cg]);
      }
    }
    if (prefetch) load_q(tnext);
    if (!(kb >= wint_lo && kb + kRChunk - 1 <= min(wint_hi, kend))) {
      const int j0 = kb + 8 * q;  // this lane's keys are kb + 8 q + e, e = 4 ab + i
#pragma unroll
      for (int cg = 0; cg < kRCG; ++cg) {
        const int lo_e = max(clo[cg] - j0, 0);
        const int hi_e = min(min(cpos[cg], kend) - j0, 7);
        const uint32_t bits = hi_e < lo_e ? 0u : ((2u << hi_e) - 1u) & ~((1u << lo_e) - 1u);
#pragma unroll
        for (int ab = 0; ab < 2; ++ab)
#pragma unroll
          for (int i = 0; i < 4; ++i) sc[ab][cg][i] = (bits >> (4 * ab + i)) & 1u ? sc[ab][cg][i] : -INFINITY;
      }
    }
    u32x4 pf[kRCG];
    float ts[kRCG];
    auto exps = [&]() {
#pragma unroll
      for (int cg = 0; cg < kRCG; ++cg) {
        float pr[8];
#pragma unroll
        for (int ab = 0; ab < 2; ++ab)
#pragma unroll
          for (int i = 0; i < 4; ++i) pr[4 * ab + i] = fast_exp2(fmaf(sc[ab][cg][i], c2, -m[cg]));
        ts[cg] = 0.f;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          pf[cg][jj] = pack_bf16x2(pr[2 * jj], pr[2 * jj + 1]);
          ts[cg] = dot2_bf16_ones(pf[cg][jj], ts[cg]);
        }
      }
    };
    bool raise = first;
    if (!first) {
      exps();
#pragma unroll
      for (int cg = 0; cg < kRCG; ++cg) raise = raise || !(ts[cg] <= kRLaneSumLimit);
    }
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
#pragma unroll
      for (int cg = 0; cg < kRCG; ++cg) {
        const float a8[8] = {sc[0][cg][0], sc[0][cg][1], sc[0][cg][2], sc[0][cg][3],
                             sc[1][cg][0], sc[1][cg][1], sc[1][cg][2], sc[1][cg][3]};
        const float cmax = max_xor32(max_xor16(max8(a8))) * c2;
        const bool up = cmax > m[cg];
        const float alpha = up ? fast_exp2(m[cg] - cmax) : 1.f;
        m[cg] = up ? cmax : m[cg];
        lsum[cg] *= alpha;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) acc[cg][dt] *= alpha;
      }
      exps();
    }
#pragma unroll
    for (int cg = 0; cg < kRCG; ++cg) lsum[cg] += ts[cg];
    // V^T operands in two batches of four (fewer registers live at once)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      u32x4 vf[4];
#pragma unroll
      for (int d4 = 0; d4 < 4; ++d4) vf[d4] = *lds128(a + kRKBytes + 1024 * (4 * h + d4));
#pragma unroll
      for (int d4 = 0; d4 < 4; ++d4)
#pragma unroll
        for (int cg = 0; cg < kRCG; ++cg)
          acc[cg][4 * h + d4] = mfma16x16x32(vf[d4], pf[cg], acc[cg][4 * h + d4]);
    }
  };

  // ---- warm-up: the chunks of the first tile, two stages in flight ----
  auto tile_last_key = [&](int t) { return P + min(C, (t + 1) * npos) - 1; };
  RStage sa, sb;
  const int ce0 = chunk_of(tile_last_key(t0));
  for (int c = 0; c <= ce0; c += 2) {
    fetch(c, sa);
    fetch(c + 1, sb);
    store(c, sa);
    if (c + 1 <= ce0) store(c + 1, sb);
  }
  int stored = ce0 + 1;  // next chunk to store
  load_q(t0);
  fetch(stored, sa);     // the chunk the next tile adds
  // Everything issued so far completes here, once: the tile loop then starts
  // with nothing pending, and the wait for each tile's queries counts only
  // the operations the previous tile issued after them (the next stage's
  // loads and the output stores), instead of waiting for those as well.
  __builtin_amdgcn_s_waitcnt(0);

  // One tile. kFull: every row of the tile is a valid position (all tiles but
  // a sequence's last); then every memory operation of the tile is issued
  // unconditionally, so the wait before the staged chunk's LDS store counts
  // exactly the operations issued after its loads and never waits for the
  // query prefetch or the output stores.
  auto tile = [&](int t, auto full_tag) {
    constexpr bool kFull = decltype(full_tag)::value;
    const int q0 = t * npos, q1 = min(C, q0 + npos) - 1;
    __syncthreads();
#pragma unroll
    for (int cg = 0; cg < kRCG; ++cg) {
      const int row = wave * (16 * kRCG) + cg * 16 + r;
      const int po = row / G;
      cval[cg] = q0 + po <= q1;
      cpos[cg] = P + q0 + po;
      clo[cg] = max(0, cpos[cg] - W + 1);
      m[cg] = -FLT_MAX;
      lsum[cg] = 0.f;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) acc[cg][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // this wave's rows: positions po_lo .. po_hi of the tile (a wave has no
    // rows only in a sequence's last, partial tile, which ends its run)
    const int po_lo = (wave * 16 * kRCG) / G;
    const int po_hi = min((wave * 16 * kRCG + 16 * kRCG - 1) / G, q1 - q0);
    const bool more = t + 1 < t1;
    if (kFull || po_lo <= q1 - q0) {
      const int wklo = max(0, P + q0 + po_lo - W + 1), wkhi = P + q0 + po_hi;
      const int wint_lo = max(0, P + q0 + po_hi - W + 1), wint_hi = P + q0 + po_lo;
      const int cw0 = chunk_of(wklo), cw1 = chunk_of(wkhi);
      // the last chunk is peeled off: only it overwrites the queries (with the
      // next tile's; on the run's last tile a harmless reload of this one), so
      // the loop keeps them in place
      for (int c = cw0; c < cw1; ++c)
        chunk(c, chunk_base(c), c < ncached ? chi : khi, wint_lo, wint_hi, c == cw0, false, 0);
      chunk(cw1, chunk_base(cw1), cw1 < ncached ? chi : khi, wint_lo, wint_hi, cw1 == cw0, true,
            more ? t + 1 : t);
    }
    // normalise this tile's rows
    u32x2 wo[kRCG][8];
#pragma unroll
    for (int cg = 0; cg < kRCG; ++cg) {
      const float l = sum_xor32(sum_xor16(lsum[cg]));
      const float inv = 1.f / l;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        wo[cg][dt][0] = pack_bf16x2(acc[cg][dt][0] * inv, acc[cg][dt][1] * inv);
        wo[cg][dt][1] = pack_bf16x2(acc[cg][dt][2] * inv, acc[cg][dt][3] * inv);
      }
    }
    // Stage the chunk the next tile adds now, before this tile's output stores
    // (its loads went out a tile ago). A tile's last key is its last query's
    // position, always a new key, and the next tile's lies at most 32
    // positions further (256 / G <= 32), so it adds at most one chunk. Its
    // buffer held a chunk that ends before this tile's range, so waves still
    // computing this tile are not disturbed; the barrier that opens the next
    // tile makes it visible. The stage is reloaded either way (with the same
    // chunk when nothing was stored), keeping the loads unconditional.
    const bool adv = more && stored <= chunk_of(tile_last_key(t + 1));
    if (adv) store(stored, sa);
    stored += adv ? 1 : 0;
    fetch(stored, sa);
    // write this tile's rows
#pragma unroll
    for (int cg = 0; cg < kRCG; ++cg) {
      const int row = wave * (16 * kRCG) + cg * 16 + r;
      const int po = row / G, head = row - po * G;
      uint16_t *orow = p.out + ((int64_t)(tok0 + q0 + (kFull || cval[cg] ? po : 0)) * hq + (int64_t)g * G + head) * kHeadDim;
      store_out_row(orow, wo[cg], q, kFull || cval[cg]);
    }
  };
  const int tfull = min(t1, C / npos);  // tiles before tfull hold npos valid positions
  int t = t0;
  for (; t < tfull; ++t) tile(t, std::true_type{});
  for (; t < t1; ++t) tile(t, std::false_type{});
}

}  // namespace

bool prefill_run_fits(const PrefillParams &p) {
  const int npos = kRRows / p.group;
  return p.group >= 8 && p.pool.window > 0 && p.pool.window + npos - 1 <= 160;
}

hipError_t launch_prefill_run(const PrefillParams &p, hipStream_t stream) {
  if (p.ns <= 0 || p.max_chunk_len <= 0 || p.total_tokens <= 0) return hipSuccess;
  const int npos = kRRows / p.group;
  const int64_t ntq = (p.max_chunk_len + npos - 1) / npos;
  const int64_t npairs = (int64_t)p.ns * p.hkv;
  const int64_t runs = std::max<int64_t>(1, std::min<int64_t>(ntq, (kRTargetGroups + npairs - 1) / npairs));
  return launch_kernel(prefill_run_kernel, dim3((unsigned)(npairs * runs)), dim3(kRThreads), stream, p);
}

}  // namespace hswa
