// Windowed (SWA) chunked prefill: the query at position p attends keys
// p - W + 1 .. p only ("Compute Analysis": an SWA layer's attention covers a
// local window, so its prefill cost is linear in the chunk and the layer is
// bound by moving q, o and the chunk's K/V, not by the matrix cores).
//
// The FULL-layer kernel (prefill.hip) is built for long key ranges: 256 query
// rows per workgroup, four 32 KiB tile buffers, one workgroup per CU. For a
// window of a few hundred keys most of its work is prologue and masked pairs.
// This kernel instead gives each workgroup 128 query rows (4 waves x 32 rows,
// a row = a (position, query head) pair of one KV head's GQA group), streams
// the workgroup's key range W + 128 / G - 1 through a ring of four 32-key
// chunk buffers (64 KiB, so two workgroups share a CU and hide each other's
// memory latency) with the global loads two chunks ahead, and lets each wave
// skip the chunks that lie wholly outside the windows of its own rows.
//
// Per 32-key chunk and wave (bf16 MFMA, fp32 accumulate):
//   S^T[key][row] = K[key][:] . Q[row][:]     (Q held in registers)
//   online softmax per row (exp2, scale * log2 e folded in, running maximum in
//   exp2 units, raised lazily as in the FULL kernel)
//   O^T[d][row]  += V^T[d][key] . P^T[key][row]
// LDS holds each chunk in MFMA operand order (K: 8 blocks of 1 KiB, block
// (ab, t) for lane r + 16 q = dims 32 t + 8 q .. +7 of chunk key
// 8 (r >> 2) + 4 ab + (r & 3), the pool's own K block layout; V^T: block dt for
// lane r + 16 q = keys 8 q .. +7 of dim 16 dt + r), so every operand read is
// one conflict-free ds_read_b128. Keys outside the workgroup's range are
// staged as zeros and every column masks its own window, so stale or NaN cache
// slots never reach an accumulator.
#include <cfloat>

#include "hswa_common.h"
#include "hswa_launch.h"

namespace hswa {
namespace {

constexpr int kWThreads = 256;
constexpr int kWWaves = kWThreads / kWave;  // 4
constexpr int kWRows = kWWaves * 32;         // query rows per workgroup
constexpr int kWChunk = 32;                  // keys per chunk
constexpr int kWBufs = 4;                    // chunks c, c + 1 ready; c + 2 being stored; c - 1 done
constexpr int kWKBytes = kWChunk * kHeadDim * 2;  // 8 KiB of K per chunk
constexpr int kWBufBytes = 2 * kWKBytes;          // K, then V^T
constexpr int kWXcds = 8;
constexpr int kWCG = 2;                    // 16-column MFMA groups per wave
constexpr float kWLaneSumLimit = 4096.f;   // lane share of a row sum that raises the maximum

struct WStage {
  u32x4 k[2], v[2];
  uint32_t keep;  // bit i: k[i] holds data (else zeros are stored); bits 8 + 8 i ..: the
                  // elements (keys) of v[i] that hold data
  bool vrow;      // v[] holds key rows (chunk keys), transposed at the store
};

__global__ __launch_bounds__(kWThreads) __attribute__((amdgpu_waves_per_eu(2))) void prefill_window_kernel(
    PrefillParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char s_lds[kWBufs * kWBufBytes];

  const PoolView &pv = p.pool;
  const int G = p.group;
  const int npos = kWRows / G;  // positions per workgroup

  // Workgroup ids go to the XCDs round-robin; (sequence, KV head) pair
  // x + 8 k runs on XCD x, its position tiles in order, so the workgroups an
  // XCD holds at once are neighbouring tiles of one pair and share their keys
  // in that XCD's L2.
  const int ntq = (p.max_chunk_len + npos - 1) / npos;
  const int npairs = p.ns * p.hkv;
  const int xcd = (int)(blockIdx.x % kWXcds);
  const int local = (int)(blockIdx.x / kWXcds);
  const int k = local / ntq;
  const int tq = local - k * ntq;
  const int pair = xcd + kWXcds * k;
  if (pair >= npairs) return;
  const int b = pair / p.hkv, g = pair - b * p.hkv;

  const int tok0 = p.cu_seqlens[b];
  const int C = min(min(p.cu_seqlens[b + 1], p.total_tokens) - tok0, p.max_chunk_len);
  const int P = p.prefix_lens[b];
  const int q0 = tq * npos;
  if (q0 >= C || P < 0 || tok0 < 0) return;
  const int q1 = min(C, q0 + npos) - 1;
  const int W = pv.window;
  const int pfirst = P + q0, plast = P + q1;
  const int klo = max(0, pfirst - W + 1), khi = plast;

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r = lane & 15, q = lane >> 4;
  const int hkv = p.hkv, hq = p.hq;
  const int shift = pv.pg_shift, pg = 1 << shift;
  const float c2 = p.scale_log2;

  // Page ids of the workgroup's cached keys: lane i holds the physical page
  // of logical page lp0 + i (-1: not cached, or not a valid page). The chunks
  // cover at most W + npos + 30 <= 670 keys from lp0's first key on: at most
  // 43 pages of 16 keys, so every cached key's page is in this table and the
  // staging never waits on a block-table load.
  const int lp0 = (klo & ~(kWChunk - 1)) >> shift;
  int tab = -1;
  {
    const int lp = lp0 + lane;
    if (P > 0 && lp <= ((min(P, khi + 1) - 1) >> shift)) {
      const int e = pv.ring > 0 ? lp % pv.ring : lp;
      if (e < pv.stride) {
        const int64_t v = pv.table[(int64_t)b * pv.stride + e];
        tab = (v >= 0 && v < pv.num_pages) ? (int)v : -1;
      }
    }
  }

  // Q^T operands and the window of each of this lane's columns.
  u32x4 qf[kWCG][4];
  int cpos[kWCG], clo[kWCG];
  bool cval[kWCG];
#pragma unroll
  for (int cg = 0; cg < kWCG; ++cg) {
    const int row = wave * (16 * kWCG) + cg * 16 + r;
    const int po = row / G, head = row - po * G;
    cval[cg] = q0 + po <= q1;
    cpos[cg] = P + q0 + po;
    clo[cg] = max(0, cpos[cg] - W + 1);
    const int64_t tok = tok0 + q0 + (cval[cg] ? po : 0);
    const uint16_t *qrow = p.q + (tok * hq + (int64_t)g * G + head) * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 v = ldg128(qrow + 32 * t + 8 * q);
      const u32x4 z = {0u, 0u, 0u, 0u};
      qf[cg][t] = cval[cg] ? v : z;
    }
  }
  // This wave's rows: positions po_lo .. po_hi of the tile (none if po_lo is
  // past the last valid one). Its keys are [wklo, wkhi]; a chunk inside
  // [wint_lo, wint_hi] is visible to every one of its columns (no mask).
  const int po_lo = (wave * 16 * kWCG) / G;
  const int po_hi = min((wave * 16 * kWCG + 16 * kWCG - 1) / G, q1 - q0);
  const bool wact = po_lo <= q1 - q0;
  const int wklo = max(klo, P + q0 + po_lo - W + 1);
  const int wkhi = min(khi, P + q0 + po_hi);
  const int wint_lo = max(0, P + q0 + po_hi - W + 1);
  const int wint_hi = P + q0 + po_lo;

  // ---- staging: global -> registers -> LDS ----
  // Thread tid stores K pieces idx = tid and tid + 256 at byte 16 idx of the
  // K block: block (ab, t) = idx >> 6, lane r + 16 qq = idx & 63, i.e. dims
  // 32 t + 8 qq .. +7 of chunk key 8 (r >> 2) + 4 ab + (r & 3). V^T pieces:
  // block dt = idx >> 6 holds for lane r + 16 qq keys 8 qq .. +7 of dim
  // 16 dt + r.
  auto k_key = [](int idx) { return ((idx & 15) >> 2) * 8 + (idx >> 8) * 4 + (idx & 3); };
  auto k_dim = [](int idx) { return ((idx >> 6) & 3) * 32 + ((idx >> 4) & 3) * 8; };
  auto v_dim = [](int idx) { return (idx >> 6) * 16 + (idx & 15); };
  auto v_keys = [](int idx) { return ((idx >> 4) & 3) * 8; };
  const u32x4 zero = {0u, 0u, 0u, 0u};
  // physical page of cached key j (-1: not cached or not valid), from the lane table
  auto page_at = [&](int j) { return __shfl(tab, (j >> shift) - lp0, kWave); };
  // The key range is cut at P into cached chunks, aligned to 32 absolute
  // positions (so that 8 consecutive keys of a V^T piece are 16 contiguous
  // bytes of one pool page), and chunks of the new keys, aligned to P. No chunk
  // holds both kinds, and every fetch is the same four 16-byte loads per thread,
  // written straight into the stage registers; pieces or keys outside the
  // range are zeroed only when the stage is stored, so a fetch never waits for
  // its own loads and a store waits only for its own stage.
  const int chi = min(P - 1, khi);  // last cached key (< klo: none)
  const int ncached = klo <= chi ? ((chi - (klo & ~(kWChunk - 1))) >> 5) + 1 : 0;
  const int nbase = max(klo, P) - P;  // first new key's offset from P
  const int nnew = khi >= max(klo, P) ? ((khi - P) >> 5) - (nbase >> 5) + 1 : 0;
  const int nch = ncached + nnew;
  auto chunk_base = [&](int c) {
    return c < ncached ? (klo & ~(kWChunk - 1)) + kWChunk * c : P + kWChunk * ((nbase >> 5) + c - ncached);
  };
  auto fetch = [&](int c, WStage &st) {
    c = min(c, nch - 1);  // past the end: a repeat of the last chunk, never stored
    const int kb = chunk_base(c);
    const uint16_t *ka[2], *va[2];
    uint32_t keep = 0u;
    if (c < ncached) {
      // cached keys, any page size: K piece = dims k_dim of one key, V^T piece =
      // keys 8 qq .. +7 (8-aligned, one page) of one dim
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int idx = tid + kWThreads * i;
        const int j = kb + k_key(idx);
        const int kpage = page_at(j);
        const bool in = j >= klo && j <= chi && kpage >= 0;
        ka[i] = pv.k_pool + k_offset(pv, in ? kpage : 0, hkv, g, j & (pg - 1), k_dim(idx));
        const int j0 = kb + v_keys(idx);
        const int vpage = page_at(j0);
        va[i] = pv.v_pool + v_offset(pv, vpage >= 0 ? vpage : 0, hkv, g, j0 & (pg - 1), v_dim(idx));
        const uint32_t kv8 = vpage >= 0 ? key_range_bits(j0, klo, chi) : 0u;
        keep |= (in ? 1u : 0u) << i;
        keep |= kv8 << (8 + 8 * i);
      }
      st.vrow = false;
    } else {
      // new keys: K rows as 16-byte pieces; V rows as 16-byte pieces of keys
      // 8 wave + 4 i + lane / 16, dims 8 (lane % 16) .. +7 (transposed at the
      // store). Keys past khi read row tok0 (in bounds) and are not kept.
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int idx = tid + kWThreads * i;
        const int j = kb + k_key(idx);
        const bool in = j >= klo && j <= khi;
        ka[i] = p.k_new + ((int64_t)(tok0 + (in ? j - P : 0)) * hkv + g) * kHeadDim + k_dim(idx);
        const int jv = kb + 8 * wave + 4 * i + (lane >> 4);
        const bool inv = jv >= klo && jv <= khi;
        va[i] = p.v_new + ((int64_t)(tok0 + (inv ? jv - P : 0)) * hkv + g) * kHeadDim + (lane & 15) * 8;
        keep |= (in ? 1u : 0u) << i;
        keep |= (inv ? 0xFFu : 0u) << (8 + 8 * i);
      }
      st.vrow = true;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      st.k[i] = ldg128_global(ka[i]);
      st.v[i] = ldg128_global(va[i]);
    }
    st.keep = keep;
  };
  auto lds128 = [&](uint32_t off) { return reinterpret_cast<u32x4 *>(s_lds + off); };
  auto buf_off = [&](int buf) { return (uint32_t)__builtin_amdgcn_readfirstlane(buf * kWBufBytes); };
  // V^T bytes of dims 8 (lane % 16) + 2 (lane / 16) and + 1, keys 8 wave .. +7
  const uint32_t st_vrow = kWKBytes + ((((8 * (lane & 15)) >> 4) * 64 + ((8 * (lane & 15) + 2 * (lane >> 4)) & 15) +
                                        16 * wave) * 16);
  // 4 x 4 transpose of dwords across the lanes l, l ^ 16, l ^ 32, l ^ 48.
  auto transpose4 = [&](const u32x4 &t, uint32_t (&w)[4]) {
    const auto a = __builtin_amdgcn_permlane32_swap(t[0], t[2], false, false);
    const auto bb = __builtin_amdgcn_permlane32_swap(t[1], t[3], false, false);
    const auto c = __builtin_amdgcn_permlane16_swap((uint32_t)a[0], (uint32_t)bb[0], false, false);
    const auto d = __builtin_amdgcn_permlane16_swap((uint32_t)a[1], (uint32_t)bb[1], false, false);
    w[0] = (uint32_t)c[0];
    w[1] = (uint32_t)c[1];
    w[2] = (uint32_t)d[0];
    w[3] = (uint32_t)d[1];
  };
  auto store = [&](int buf, const WStage &st0) {
    WStage st = st0;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      st.k[i] = (st.keep >> i) & 1u ? st.k[i] : zero;
      const uint32_t kv8 = (st.keep >> (8 + 8 * i)) & 0xFFu;
      if (kv8 != 0xFFu) st.v[i] = keep_bf16x8(st.v[i], kv8);
    }
    const uint32_t bo = buf_off(buf);
    *lds128(bo + 16 * tid) = st.k[0];
    *lds128(bo + 16 * (tid + kWThreads)) = st.k[1];
    if (!st.vrow) {
      *lds128(bo + kWKBytes + 16 * tid) = st.v[0];
      *lds128(bo + kWKBytes + 16 * (tid + kWThreads)) = st.v[1];
    } else {
      // lanes l % 16 + 16 m hold keys 8 wave + 4 i + m (piece i) x dims
      // 8 (l % 16) .. +7; after the transposes lane m holds dims 2 m, 2 m + 1
      // of keys 8 wave .. +7, split into one V^T piece per dim
      uint32_t w[8];
      transpose4(st.v[0], *reinterpret_cast<uint32_t(*)[4]>(&w[0]));
      transpose4(st.v[1], *reinterpret_cast<uint32_t(*)[4]>(&w[4]));
      u32x4 lo, hi;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        lo[j] = __builtin_amdgcn_perm(w[2 * j + 1], w[2 * j], 0x05040100u);
        hi[j] = __builtin_amdgcn_perm(w[2 * j + 1], w[2 * j], 0x07060302u);
      }
      *lds128(bo + st_vrow) = lo;
      *lds128(bo + st_vrow + 16) = hi;
    }
  };

  float m[kWCG], lsum[kWCG];  // m: running maximum in exp2 units
  f32x4 acc[kWCG][8];
#pragma unroll
  for (int cg = 0; cg < kWCG; ++cg) {
    m[cg] = -FLT_MAX;
    lsum[cg] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[cg][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const uint32_t op_lane = lane * 16;
  // One chunk: QK^T, masks, online softmax, PV. The exponentials are taken
  // against the running maximum as it stands; only if some lane's share of a
  // row sum (8 probabilities) exceeds 2^12 (an infinite one included) is the
  // exact column maximum formed, the maximum raised, the output and row sum
  // rescaled and the exponentials taken again (exact either way: numerator and
  // denominator share the maximum).
  auto chunk = [&](int buf, int kb, int kend) {  // kend: the chunk's last key that holds data
    const uint32_t a = buf_off(buf) + op_lane;
    f32x4 sc[2][kWCG];
#pragma unroll
    for (int ab = 0; ab < 2; ++ab)
#pragma unroll
      for (int cg = 0; cg < kWCG; ++cg) sc[ab][cg] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 ka = *lds128(a + 1024 * t);
      const u32x4 kbv = *lds128(a + 4096 + 1024 * t);
#pragma unroll
      for (int cg = 0; cg < kWCG; ++cg) {
        sc[0][cg] = mfma16x16x32(ka, qf[cg][t], sc[0][cg]);
        sc[1][cg] = mfma16x16x32(kbv, qf[cg][t], sc[1][cg]);
      }
    }
    // V^T operands, read while the scores are formed
    u32x4 vf[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) vf[dt] = *lds128(a + kWKBytes + 1024 * dt);
    if (!(kb >= wint_lo && kb + kWChunk - 1 <= min(wint_hi, kend))) {
      // this lane's keys are kb + 8 q + e, e = 4 ab + i
      const int j0 = kb + 8 * q;
#pragma unroll
      for (int cg = 0; cg < kWCG; ++cg) {
        const int lo_e = max(clo[cg] - j0, 0);
        const int hi_e = min(min(cpos[cg], kend) - j0, 7);
        const uint32_t bits = hi_e < lo_e ? 0u : ((2u << hi_e) - 1u) & ~((1u << lo_e) - 1u);
#pragma unroll
        for (int ab = 0; ab < 2; ++ab)
#pragma unroll
          for (int i = 0; i < 4; ++i) sc[ab][cg][i] = (bits >> (4 * ab + i)) & 1u ? sc[ab][cg][i] : -INFINITY;
      }
    }
    u32x4 pf[kWCG];
    float ts[kWCG];
    auto exps = [&]() {
#pragma unroll
      for (int cg = 0; cg < kWCG; ++cg) {
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
    exps();
    bool raise = false;
#pragma unroll
    for (int cg = 0; cg < kWCG; ++cg) raise = raise || !(ts[cg] <= kWLaneSumLimit);
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
#pragma unroll
      for (int cg = 0; cg < kWCG; ++cg) {
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
    for (int cg = 0; cg < kWCG; ++cg) lsum[cg] += ts[cg];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
      for (int cg = 0; cg < kWCG; ++cg) acc[cg][dt] = mfma16x16x32(vf[dt], pf[cg], acc[cg][dt]);
  };

  // ---- chunk loop: chunk c is computed from buffer c % 4. Two register
  // stages carry the global loads two chunks ahead: chunk c + 2, loaded during
  // chunk c - 2 (or before the loop), is stored into buffer (c + 2) % 4 after
  // chunk c's compute (chunk c - 2 read that buffer, and the barrier that
  // opens chunk c - 1 ended those reads), and chunk c + 4's loads go out into
  // the stage it frees.
  // Every step issues the same loads (one fetch), so that the wait before a
  // stage's store counts exactly the other stage's loads.
  WStage st[2];
  fetch(0, st[0]);
  fetch(1, st[1]);
  store(0, st[0]);
  fetch(2, st[0]);
  if (nch > 1) store(1, st[1]);
  fetch(3, st[1]);
  auto step = [&](int c, WStage &s2) {  // s2: the stage holding chunk c + 2
    const int kb = chunk_base(min(c, nch - 1));
    __syncthreads();
    if (c < nch && wact && kb + kWChunk - 1 >= wklo && kb <= wkhi) chunk(c % kWBufs, kb, c < ncached ? chi : khi);
    if (c + 2 < nch) store((c + 2) % kWBufs, s2);
    fetch(c + 4, s2);
  };
  // unrolled by two, both steps unconditional (a step past the end only
  // fetches), so each stage is named statically and the newest loads are
  // always the other stage's
  for (int c = 0; c < nch; c += 2) {
    step(c, st[0]);
    step(c + 1, st[1]);
  }

  // ---- normalise and write ----
#pragma unroll
  for (int cg = 0; cg < kWCG; ++cg) {
    const float l = sum_xor32(sum_xor16(lsum[cg]));
    const float inv = 1.f / l;
    const int row = wave * (16 * kWCG) + cg * 16 + r;
    const int po = row / G, head = row - po * G;
    uint16_t *orow = p.out + ((int64_t)(tok0 + q0 + (cval[cg] ? po : 0)) * hq + (int64_t)g * G + head) * kHeadDim;
    u32x2 w[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      w[dt][0] = pack_bf16x2(acc[cg][dt][0] * inv, acc[cg][dt][1] * inv);
      w[dt][1] = pack_bf16x2(acc[cg][dt][2] * inv, acc[cg][dt][3] * inv);
    }
    store_out_row(orow, w, q, cval[cg]);
  }
}

}  // namespace

hipError_t launch_prefill_window(const PrefillParams &p, hipStream_t stream) {
  if (p.ns <= 0 || p.max_chunk_len <= 0 || p.total_tokens <= 0) return hipSuccess;
  const int npos = kWRows / p.group;
  const int64_t ntq = (p.max_chunk_len + npos - 1) / npos;
  const int64_t pairs_per_xcd = ((int64_t)p.ns * p.hkv + kWXcds - 1) / kWXcds;
  const int64_t grid = pairs_per_xcd * ntq * kWXcds;
  return launch_kernel(prefill_window_kernel, dim3((unsigned)grid), dim3(kWThreads), stream, p);
}

}  // namespace hswa
