// Chunked prefill attention over a cached prefix.
//
// "Compute Analysis": chunked prefill is largely compute-bound, and an SWA
// layer only needs the keys inside its window, so tiles outside the window are
// never visited. Keys below the prefix length P come from the paged cache (FULL:
// the block table; SWA: the ring), keys from P on come from the chunk's own
// k_new / v_new (the chunk is appended to the cache only after this kernel).
//
// Work unit: one workgroup (4 waves) per (tile of 128 query rows, KV head,
// sequence). A query row is a (position, query head) pair of the KV head's GQA
// group, so one K/V tile in LDS serves every query head that shares it. Each
// wave owns 32 rows (two 16-column MFMA groups). Per 64-key tile:
//   S^T[key][row]  = K[key][:] . Q[row][:]          (bf16 MFMA, fp32 accumulate)
//   online softmax per row in fp32 (exp2, scale*log2(e) folded in)
//   O^T[d][row]   += V^T[d][key] . P^T[key][row]    (bf16 MFMA)
// K is staged in LDS as rows, V as its transpose, both XOR-swizzled so that the
// 16 lanes reading one MFMA operand hit distinct banks. Keys outside the
// workgroup's range are staged as zeros, so NaN or stale data in unused cache
// slots never reaches an accumulator; per-element masks are applied only on
// tiles that cross the causal diagonal, the window edge or the range ends.
#include "hswa_common.h"
#include "hswa_launch.h"

namespace hswa {
namespace {

constexpr int kThreads = 256;
constexpr int kRows = 128;  // query rows per workgroup
constexpr int kKT = 64;     // keys per tile

__device__ __forceinline__ int swz_k(int key) { return (key & 3) | (((key >> 3) & 3) << 2); }

__device__ __forceinline__ int64_t prefix_page(const PoolView &pv, int b, int key, bool &ok) {
  int lp = key >> pv.pg_shift;
  if (pv.ring > 0) lp %= pv.ring;
  if (lp >= pv.stride) {
    ok = false;
    return 0;
  }
  const int64_t page = pv.table[(int64_t)b * pv.stride + lp];
  ok = page >= 0 && page < pv.num_pages;
  return ok ? page : 0;
}

__global__ __launch_bounds__(kThreads) void prefill_kernel(PrefillParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t s_k[kKT * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t s_v[kHeadDim * kKT];

  const PoolView &pv = p.pool;
  const int b = blockIdx.z, g = blockIdx.y;
  const int G = p.group;
  const int npos = kRows / G;  // positions per workgroup
  const int tok0 = p.cu_seqlens[b];
  // never step outside q / k_new / v_new / out, whatever the device offsets say
  const int C = min(min(p.cu_seqlens[b + 1], p.total_tokens) - tok0, p.max_chunk_len);
  const int P = p.prefix_lens[b];
  const int q0 = blockIdx.x * npos;
  if (q0 >= C || P < 0 || tok0 < 0) return;
  const int q1 = min(C, q0 + npos) - 1;
  const int pfirst = P + q0, plast = P + q1;
  const int W = pv.window;
  const int klo = W > 0 ? max(0, pfirst - W + 1) : 0;
  const int khi = plast;

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int r = lane & 15, q = lane >> 4;
  const int hkv = p.hkv, hq = p.hq;
  const int shift = pv.pg_shift, pg = 1 << shift;
  const float c2 = p.scale_log2;

  // Q^T operands and the position of each of this lane's two columns.
  u32x4 qf[2][4];
  int cpos[2], clo[2];
  bool cval[2];
#pragma unroll
  for (int cg = 0; cg < 2; ++cg) {
    const int row = wave * 32 + cg * 16 + r;
    const int po = row / G, head = row - po * G;
    cval[cg] = q0 + po <= q1;
    cpos[cg] = P + q0 + po;
    clo[cg] = W > 0 ? max(0, cpos[cg] - W + 1) : 0;
    const int64_t tok = tok0 + q0 + (cval[cg] ? po : 0);
    const uint16_t *qrow = p.q + (tok * hq + (int64_t)g * G + head) * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 v = ldg128(qrow + 32 * t + 8 * q);
      const u32x4 z = {0u, 0u, 0u, 0u};
      qf[cg][t] = cval[cg] ? v : z;
    }
  }

  float m[2] = {-INFINITY, -INFINITY}, lsum[2] = {0.f, 0.f};
  f32x4 acc[2][8];
#pragma unroll
  for (int cg = 0; cg < 2; ++cg)
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[cg][dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kt = klo & ~(kKT - 1); kt <= khi; kt += kKT) {
    __syncthreads();  // the previous tile has been consumed
    // ---- stage K rows ----
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + kThreads * i;
      const int key = idx >> 4, c = idx & 15;
      const int j = kt + key;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (j >= klo && j <= khi) {
        if (j < P) {
          bool ok;
          const int64_t page = prefix_page(pv, b, j, ok);
          if (ok) v = ldg128(pv.k_pool + (((page * hkv + g) << shift) + (j & (pg - 1))) * kHeadDim + c * 8);
        } else {
          v = ldg128(p.k_new + ((int64_t)(tok0 + j - P) * hkv + g) * kHeadDim + c * 8);
        }
      }
      *reinterpret_cast<u32x4 *>(s_k + key * kHeadDim + ((c ^ swz_k(key)) * 8)) = v;
    }
    // ---- stage V^T ----
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + kThreads * i;
      const int d = idx >> 3, kc = idx & 7;
      const int j0 = kt + 8 * kc;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (j0 >= klo && j0 + 7 <= khi && j0 + 7 < P) {
        bool ok;
        const int64_t page = prefix_page(pv, b, j0, ok);
        if (ok) v = ldg128(pv.v_pool + ((page * hkv + g) * kHeadDim + d) * pg + (j0 & (pg - 1)));
      } else if (j0 + 7 >= klo && j0 <= khi) {
        uint32_t e[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int j = j0 + t;
          e[t] = 0u;
          if (j >= klo && j <= khi) {
            if (j < P) {
              bool ok;
              const int64_t page = prefix_page(pv, b, j, ok);
              if (ok) e[t] = pv.v_pool[((page * hkv + g) * kHeadDim + d) * pg + (j & (pg - 1))];
            } else {
              e[t] = p.v_new[((int64_t)(tok0 + j - P) * hkv + g) * kHeadDim + d];
            }
          }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = e[2 * t] | (e[2 * t + 1] << 16);
      }
      *reinterpret_cast<u32x4 *>(s_v + d * kKT + ((kc ^ (d & 7)) * 8)) = v;
    }
    __syncthreads();

    // ---- S^T = K Q^T ----
    float s[2][2][8];  // [half][cg][key]
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      u32x4 ka[4], kb[4];
      const int keya = 32 * h + 8 * (r >> 2) + (r & 3);
      const int keyb = keya + 4;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int c = 4 * t + q;
        ka[t] = *reinterpret_cast<const u32x4 *>(s_k + keya * kHeadDim + ((c ^ swz_k(keya)) * 8));
        kb[t] = *reinterpret_cast<const u32x4 *>(s_k + keyb * kHeadDim + ((c ^ swz_k(keyb)) * 8));
      }
#pragma unroll
      for (int cg = 0; cg < 2; ++cg) {
        f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          sa = mfma16x16x32(ka[t], qf[cg][t], sa);
          sb = mfma16x16x32(kb[t], qf[cg][t], sb);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          s[h][cg][i] = sa[i];
          s[h][cg][4 + i] = sb[i];
        }
      }
    }

    // ---- masks (only on tiles that need them) ----
    const bool need_mask = kt + kKT - 1 > pfirst || kt < klo || kt + kKT - 1 > khi ||
                           (W > 0 && kt < plast - W + 1);
    if (need_mask) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int cg = 0; cg < 2; ++cg)
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int j = kt + 32 * h + 8 * q + i;
            const bool ok = j <= cpos[cg] && j >= clo[cg] && j >= klo && j <= khi;
            s[h][cg][i] = ok ? s[h][cg][i] : -INFINITY;
          }
    }

    // ---- online softmax and O^T += V^T P^T ----
    u32x4 pf[2][2];
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) {
      float cmax = -INFINITY;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 8; ++i) cmax = fmaxf(cmax, s[h][cg][i]);
      cmax = wave_max_xor(cmax, 16);
      cmax = wave_max_xor(cmax, 32);
      const float mnew = fmaxf(m[cg], cmax);
      const float mc = mnew == -INFINITY ? 0.f : mnew * c2;
      const float alpha = fast_exp2(m[cg] * c2 - mc);
      float psum = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float pr[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          pr[i] = fast_exp2(fmaf(s[h][cg][i], c2, -mc));
          psum += pr[i];
        }
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) pf[h][cg][jj] = pack_bf16x2(pr[2 * jj], pr[2 * jj + 1]);
      }
      lsum[cg] = lsum[cg] * alpha + psum;
      m[cg] = mnew;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) acc[cg][dt] *= alpha;
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int kc = 4 * h + q;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const int d = 16 * dt + r;
        const u32x4 vf = *reinterpret_cast<const u32x4 *>(s_v + d * kKT + ((kc ^ (d & 7)) * 8));
#pragma unroll
        for (int cg = 0; cg < 2; ++cg) acc[cg][dt] = mfma16x16x32(vf, pf[h][cg], acc[cg][dt]);
      }
    }
  }

  // ---- normalise and write ----
#pragma unroll
  for (int cg = 0; cg < 2; ++cg) {
    float l = wave_sum_xor(lsum[cg], 16);
    l = wave_sum_xor(l, 32);
    if (!cval[cg]) continue;
    const float inv = 1.f / l;
    const int row = wave * 32 + cg * 16 + r;
    const int po = row / G, head = row - po * G;
    uint16_t *orow = p.out + ((int64_t)(tok0 + q0 + po) * hq + (int64_t)g * G + head) * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      u32x2 w;
      w[0] = pack_bf16x2(acc[cg][dt][0] * inv, acc[cg][dt][1] * inv);
      w[1] = pack_bf16x2(acc[cg][dt][2] * inv, acc[cg][dt][3] * inv);
      *reinterpret_cast<u32x2 *>(orow + 16 * dt + 4 * q) = w;
    }
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillParams &p, hipStream_t stream) {
  if (p.ns <= 0 || p.max_chunk_len <= 0 || p.total_tokens <= 0) return hipSuccess;
  const int npos = kRows / p.group;
  const dim3 grid((p.max_chunk_len + npos - 1) / npos, p.hkv, p.ns);
  return launch_kernel(prefill_kernel, grid, dim3(kThreads), stream, p);
}

}  // namespace hswa
