// Row-batched attention over a shared prefix plus each row's own tokens.
//
// Every row r of a batch attends to the keys of its prefix chain (a root
// and optionally a child prefix, stored once per prefix and shared by all
// rows that use it) followed by its own keys, causally.  Query head j reads
// key/value head j / G (grouped-query attention, G = n_heads / n_kv_heads).
//
// Workgroup = one (row, 64-query-vector tile, kv head); a query vector is a
// (token, head-in-group) pair, so the G heads that share a kv head share
// every K/V tile read.  Keys are walked in blocks of 32 staged in LDS (K
// row-major, V transposed) and shared by the 4 waves; each wave owns 16
// query vectors and keeps an online softmax (running max and sum in fp32,
// base-2 exponent) with the scores computed transposed, S^T = K Q^T, so the
// MFMA result layout of P^T is directly the B operand of O^T = V^T P^T and
// every lane holds values of exactly one query.
#include "common.h"
#include "kernels.h"

namespace lmop {

namespace {

constexpr int KB = 32;  // keys per block

template <int HD>
__global__ __launch_bounds__(256) void attn_kernel(const AttnArgs p, float scale_log2) {
  constexpr int KS = HD + 8;   // K row stride in LDS (halves)
  constexpr int VS = KB + 8;   // V^T row stride in LDS (halves)
  constexpr int NS = HD / 32;  // k-steps of the score MFMA
  constexpr int NT = HD / 16;  // 16-dim output tiles
  __shared__ f16 sK[KB * KS];
  __shared__ f16 sV[HD * VS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int2 wk = p.work[blockIdx.x];
  const AttnRow row = p.rows[wk.x];
  const int h = blockIdx.y;  // kv head
  const int G = p.nq / p.nkv;
  const int kvdim = p.nkv * HD;
  const int P = row.seg_n[0] + row.seg_n[1];

  // this lane's query vector
  const int v = wk.y * 64 + wave * 16 + c;
  const int t = v / G;
  const bool qvalid = t < row.n_q;
  const int hq = h * G + (v - t * G);
  const int n_vis = qvalid ? P + row.own_q0 + t + 1 : 1;

  // keys needed by the workgroup: up to its last valid token
  int t_last = (wk.y * 64 + 63) / G;
  if (t_last > row.n_q - 1) t_last = row.n_q - 1;
  const int n_keys = P + row.own_q0 + t_last + 1;

  f16x8 qf[NS];
  if (qvalid) {
    const f16* qp = (const f16*)p.q + (size_t)(row.q_start + t) * p.ldq + hq * HD;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = *(const f16x8*)(qp + s * 32 + g * 8);
  } else {
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = f16x8{0, 0, 0, 0, 0, 0, 0, 0};
  }

  f32x4 o[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -1e30f, l_run = 0.f;

  const size_t own_layer = (size_t)p.layer * 2 * p.own_cap * kvdim;
  for (int kb = 0; kb < n_keys; kb += KB) {
    __syncthreads();
    // stage K (row-major) and V (transposed) of keys kb .. kb+31
    for (int ch = tid; ch < KB * HD / 8; ch += 256) {
      const int kl = ch / (HD / 8), d0 = (ch - kl * (HD / 8)) * 8;
      const int kk = kb + kl;
      f16x8 kv = f16x8{0, 0, 0, 0, 0, 0, 0, 0}, vv = kv;
      if (kk < n_keys) {
        const f16* base;
        size_t voff;
        if (kk < row.seg_n[0]) {
          const int n = row.seg_n[0];
          base = (const f16*)row.seg_kv[0] + (size_t)p.layer * 2 * n * kvdim + (size_t)kk * kvdim;
          voff = (size_t)n * kvdim;
        } else if (kk < P) {
          const int n = row.seg_n[1];
          base = (const f16*)row.seg_kv[1] + (size_t)p.layer * 2 * n * kvdim +
                 (size_t)(kk - row.seg_n[0]) * kvdim;
          voff = (size_t)n * kvdim;
        } else {
          base = (const f16*)p.own_kv + own_layer + (size_t)(row.own_slot + kk - P) * kvdim;
          voff = (size_t)p.own_cap * kvdim;
        }
        base += h * HD + d0;
        kv = *(const f16x8*)base;
        vv = *(const f16x8*)(base + voff);
      }
      *(f16x8*)(sK + kl * KS + d0) = kv;
#pragma unroll
      for (int e = 0; e < 8; ++e) sV[(d0 + e) * VS + kl] = vv[e];
    }
    __syncthreads();

    // S^T for keys kb + 16*half + (4g + r), query c
    f32x4 st[2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      st[hf] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const f16x8 a = *(const f16x8*)(sK + (hf * 16 + c) * KS + s * 32 + g * 8);
        st[hf] = mfma16x16x32(a, qf[s], st[hf]);
      }
    }
    float mb = -INFINITY;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kk = kb + hf * 16 + 4 * g + r;
        const float sc = kk < n_vis ? st[hf][r] * scale_log2 : -INFINITY;
        st[hf][r] = sc;
        mb = fmaxf(mb, sc);
      }
    mb = fmaxf(mb, shfl_xor(mb, 16));
    mb = fmaxf(mb, shfl_xor(mb, 32));
    const float m_new = fmaxf(m_run, mb);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    f16x8 pb;
    float ps = 0.f;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float e = exp2f(st[hf][r] - m_new);
        ps += e;
        pb[hf * 4 + r] = (f16)e;
      }
    l_run = l_run * alpha + ps;
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      o[i] *= alpha;
      // A = V^T rows 16i + c, keys matching P^T's register order
      const f16x4 lo = *(const f16x4*)(sV + (16 * i + c) * VS + 4 * g);
      const f16x4 hi = *(const f16x4*)(sV + (16 * i + c) * VS + 16 + 4 * g);
      const f16x8 a = f16x8{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      o[i] = mfma16x16x32(a, pb, o[i]);
    }
  }

  float l_tot = l_run + shfl_xor(l_run, 16);
  l_tot += shfl_xor(l_tot, 32);
  if (qvalid) {
    const float inv = 1.0f / l_tot;
    f16* op = (f16*)p.out + (size_t)(row.q_start + t) * p.ldo + hq * HD;
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      f16x4 w = {(f16)(o[i][0] * inv), (f16)(o[i][1] * inv), (f16)(o[i][2] * inv),
                 (f16)(o[i][3] * inv)};
      *(f16x4*)(op + 16 * i + 4 * g) = w;
    }
  }
}

}  // namespace

hipError_t launch_attention(hipStream_t s, const AttnArgs& a) {
  if (a.n_work == 0) return hipSuccess;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)a.hd);
  dim3 grid(a.n_work, a.nkv);
  if (a.hd == 128)
    hipLaunchKernelGGL(attn_kernel<128>, grid, dim3(256), 0, s, a, scale_log2);
  else if (a.hd == 64)
    hipLaunchKernelGGL(attn_kernel<64>, grid, dim3(256), 0, s, a, scale_log2);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace lmop
