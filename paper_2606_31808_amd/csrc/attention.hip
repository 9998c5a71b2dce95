// Row-batched attention over a shared prefix plus each row's own tokens.
//
// Every row of a batch attends to the keys of its prefix chain (a root and
// optionally a child prefix, each stored once and shared by all rows that
// use it) followed by its own keys, causally.  Query head j reads key/value
// head j / G (grouped-query attention, G = n_heads / n_kv_heads).
//
// KV store layout (per layer, capacity C slots, C a multiple of 64):
//   K   [C][n_kv][hd]      (row-major per token)
//   V^T [n_kv][hd][C]      (transposed, so a 64-key tile of one head is 128-byte rows)
// so that both tiles copy into LDS with direct global->LDS loads and the
// P.V product reads V^T rows with no transposition in the kernel.
//
// Workgroup = one (row, 128-query-vector tile, kv head); a query vector is
// a (token, head-in-group) pair, so the G heads sharing a kv head share all
// K/V tile reads.  Keys are walked segment by segment (root prefix, child
// prefix, own) in blocks of 64 through a two-stage LDS ring (one barrier per
// block: the next block's loads are issued right after it).  Each wave owns
// 16 (hd 128) or 32 (hd 64) query vectors and keeps an online softmax (fp32
// reference maximum and
// sum, base-2 exponent); the reference maximum moves only when a score
// exceeds it by a wide margin, so the running output is rarely rescaled.
// Waves whose query vectors all lie past the row's end only help load.  Scores are computed transposed, S^T = K Q^T, so
// the MFMA result layout of P^T is directly the B operand of O^T = V^T P^T
// and every lane holds values of exactly one query.
#include "common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace lmop {

namespace {

constexpr int KB = 64;   // keys per block
constexpr int QT = ATTN_QTILE;  // query vectors per workgroup
// waves per workgroup: with hd = 128, 8 waves of 16 query vectors (4 waves
// per SIMD hide more of each block's score -> softmax -> P.V chain than 4
// waves of 32; measured 6% faster); with hd = 64 a wave's block is already
// short, and 4 waves of 32 are 6% faster
template <int HD>
constexpr int attn_waves() { return HD == 128 ? 8 : 4; }

// Key order inside a 32-key chunk: score tile hf (0, 1) row m = 4a + b
// (a, b in 0..3) holds key 8a + 4hf + b, so that the MFMA result layout puts
// keys 8g .. 8g+7 in the registers of lane group g and the P.V operand reads
// one contiguous 16-byte run of a V^T row.
LMOP_DEVICE int score_key(int hf, int m) { return 8 * (m >> 2) + 4 * hf + (m & 3); }

// 16-byte chunk swizzles (conflict-free fragment loads on gfx950, measured
// with SQ_LDS_BANK_CONFLICT): K rows by key, V^T rows by dim
template <int HD>
LMOP_DEVICE int kswz(int key) {
  const int s = ((key >> 1) & 12) | (key & 3);  // = m of score_key within a tile
  return HD == 128 ? s : (s & 7);
}
LMOP_DEVICE int vswz(int row) { return row & 7; }


// max / sum with the lane 16 (32) apart: the gfx950 row-swap instructions
// exchange 16-lane rows between two registers without going through LDS
LMOP_DEVICE float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));  // inputs are never NaN
  return r;
}
LMOP_DEVICE float max_x16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
LMOP_DEVICE float max_x32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
LMOP_DEVICE float sum_x16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
LMOP_DEVICE float sum_x32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int HD>
__global__ __launch_bounds__(64 * attn_waves<HD>(), 2) void attn_kernel(const AttnArgs p,
                                                                         float scale_log2) {
  constexpr int NWV = attn_waves<HD>();
  constexpr int QW = QT / NWV;  // query vectors per wave
  constexpr int QS = QW / 16;   // 16-vector query sub-tiles per wave
  constexpr int K_BYTES = KB * HD * 2;
  constexpr int V_BYTES = HD * KB * 2;
  constexpr int STAGE = K_BYTES + V_BYTES;
  constexpr int K_LOADS = K_BYTES / 1024 / NWV;  // per wave
  constexpr int V_LOADS = V_BYTES / 1024 / NWV;
  constexpr int NS = HD / 32;  // k-steps of the score MFMA
  constexpr int NT = HD / 16;  // 16-dim output tiles
  constexpr int KCH = HD / 8;  // 16-byte chunks per K row
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int g = lane >> 4, c = lane & 15;
  const int2 wk = p.work[blockIdx.x];
  const AttnRow row = p.rows[wk.x];
  const int h = blockIdx.y;  // kv head
  const int G = p.nq / p.nkv;
  const int kvdim = p.nkv * HD;

  // segments: root prefix, child prefix, own tokens
  int t_last = (wk.y * QT + QT - 1) / G;
  if (t_last > row.n_q - 1) t_last = row.n_q - 1;
  // segment s: keys [start, start + n) of a store with capacity cap (K at
  // kb_s, V^T at vb_s).  Separate named scalars, chosen with selects: an
  // array indexed by the runtime segment number would live in scratch memory.
  const int cap0 = row.seg_cap[0], cap1 = row.seg_cap[1], cap2 = p.own_cap;
  const f16* kb0 = (const f16*)row.seg_kv[0] + (size_t)p.layer * 2 * cap0 * kvdim;
  const f16* kb1 = (const f16*)row.seg_kv[1] + (size_t)p.layer * 2 * cap1 * kvdim;
  const f16* kb2 = (const f16*)p.own_kv + (size_t)p.layer * 2 * cap2 * kvdim;
  const f16* vb0 = kb0 + (size_t)cap0 * kvdim;
  const f16* vb1 = kb1 + (size_t)cap1 * kvdim;
  const f16* vb2 = kb2 + (size_t)cap2 * kvdim;
  const int start0 = row.seg_start[0], start1 = row.seg_start[1], start2 = row.own_slot;
  const int n0 = row.seg_n[0], n1 = row.seg_n[1], n2 = row.own_q0 + t_last + 1;
  // own keys visible to every valid query of the workgroup (first token's count)
  int t_first = (wk.y * QT) / G;
  const int vis_min = row.own_q0 + t_first + 1;
  const int nb0 = (n0 + KB - 1) / KB, nb1 = (n1 + KB - 1) / KB;
  const int nb2 = (n2 + KB - 1) / KB;
  const int NB = nb0 + nb1 + nb2;

  // Each load's address = a block base in scalar registers + a per-lane byte
  // offset.  K offsets do not depend on the block; V^T offsets depend on the
  // segment's capacity (row stride) only.
  uint32_t koff[K_LOADS], vdim[V_LOADS], vchunk[V_LOADS];
#pragma unroll
  for (int i = 0; i < K_LOADS; ++i) {
    const int q = wave + NWV * i;  // 1 KB = 1024 / (2*HD) keys
    const int key = q * (512 / HD) + lane / KCH;
    const int chunk = (lane % KCH) ^ kswz<HD>(key);
    koff[i] = (uint32_t)(key * kvdim + h * HD + chunk * 8) * 2u;
  }
#pragma unroll
  for (int i = 0; i < V_LOADS; ++i) {
    const int q = wave + NWV * i;  // 8 dim rows of 128 bytes
    const int dim = q * 8 + (lane >> 3);
    vdim[i] = (uint32_t)dim;
    vchunk[i] = (uint32_t)(((lane & 7) ^ vswz(dim)) * 16);
  }
  // The non-empty segments in walk order, as up to three slots (a, b, c)
  // that shift down when a segment is used up: no runtime segment index
  // (it would turn the selects into a scratch-memory table).  Each slot:
  // first block's K and V^T bases (bytes), V^T row length (bytes), keys,
  // whether it is the own segment.
  struct Seg {
    const char* k;
    const char* v;
    uint32_t vrow;
    int n;
    bool own;
  };
  auto make_seg = [&](const f16* kb, const f16* vb, int cap, int start, int n, bool own) {
    return Seg{(const char*)(kb + (size_t)start * kvdim),
               (const char*)(vb + (size_t)h * HD * cap + start), (uint32_t)cap * 2u, n, own};
  };
  const Seg s0 = make_seg(kb0, vb0, cap0, start0, n0, false);
  const Seg s1 = make_seg(kb1, vb1, cap1, start1, n1, false);
  const Seg s2 = make_seg(kb2, vb2, cap2, start2, n2, true);  // never empty
  const Seg none = Seg{nullptr, nullptr, 0u, 0, true};
  Seg la = n0 > 0 ? s0 : n1 > 0 ? s1 : s2;
  Seg lb = n0 > 0 ? (n1 > 0 ? s1 : s2) : n1 > 0 ? s2 : none;
  Seg lc = n0 > 0 && n1 > 0 ? s2 : none;
  // the loads' walk: slot la holds the next block to load, lkb its first key
  int lkb = 0;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_ptr_t)smem + (uint32_t)wave * 1024u;
  auto issue = [&](int st) {
    const uint32_t mk = lds0 + (uint32_t)(st * STAGE);
#pragma unroll
    for (int i = 0; i < K_LOADS; ++i) g2l16_m0(la.k, koff[i], mk + 1024u * NWV * i);
#pragma unroll
    for (int i = 0; i < V_LOADS; ++i)
      g2l16_m0(la.v, __umul24(vdim[i], la.vrow) + vchunk[i], mk + K_BYTES + 1024u * NWV * i);
    lkb += KB;
    la.k += (size_t)KB * kvdim * 2;
    la.v += KB * 2;
    if (lkb >= la.n) {
      lkb = 0;
      la = lb;
      lb = lc;
    }
  };

  // this lane's query vectors: v = tile*128 + wave*QW + 16*qs + c
  f16x8 qf[QS][NS];
  int n_vis[QS];  // own keys visible to the query (prefix keys are all visible)
  bool qvalid[QS];
  int tok[QS], hq[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int v = wk.y * QT + wave * QW + 16 * qs + c;
    const int t = v / G;
    qvalid[qs] = t < row.n_q;
    tok[qs] = t;
    hq[qs] = h * G + (v - t * G);
    n_vis[qs] = qvalid[qs] ? row.own_q0 + t + 1 : 1;
    if (qvalid[qs]) {
      const f16* qp = (const f16*)p.q + (size_t)(row.q_start + t) * p.ldq + hq[qs] * HD;
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[qs][s] = *(const f16x8*)(qp + s * 32 + g * 8);
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[qs][s] = f16x8{0, 0, 0, 0, 0, 0, 0, 0};
    }
  }

  f32x4 o[QS][NT];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs)
#pragma unroll
    for (int i = 0; i < NT; ++i) o[qs][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[QS], l_run[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) m_run[qs] = -1e30f, l_run[qs] = 0.f;
  const float thr = 8.0f / scale_log2;

  // a wave whose query vectors all lie past the row's end only helps load
  const bool wave_active = wk.y * QT + wave * QW < row.n_q * G;
  // the computation's walk over the same blocks: keys and kind of the
  // current segment and of the ones after it, ckb the block's first key
  int ca_n = la.n, cb_n = lb.n, cc_n = lc.n;
  bool ca_own = la.own, cb_own = lb.own, cc_own = lc.own;
  int ckb = 0;
  issue(0);
  for (int b = 0; b < NB; ++b) {
    // block b is in LDS for every wave, and every wave is done with block
    // b-1, whose stage the next issue refills
    wait_vmcnt<0>();
    barrier();
    if (b + 1 < NB) issue((b + 1) & 1);
    const int seg_n = ca_n;
    const int kb_cur = ckb;
    const bool own_cur = ca_own;
    ckb += KB;
    if (ckb >= ca_n) {
      ckb = 0;
      ca_n = cb_n;
      ca_own = cb_own;
      cb_n = cc_n;
      cb_own = cc_own;
    }
    if (!wave_active) continue;
    const char* sK = smem + (b & 1) * STAGE;
    const char* sV = sK + K_BYTES;

    // S^T tiles kt = 2*kc + hf: register r of lane group g holds key
    // kb + 32*kc + 8g + 4hf + r, query (qs, c)
    f32x4 st[QS][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      f16x8 a[NS];
      const int key = 32 * (kt >> 1) + score_key(kt & 1, c);
#pragma unroll
      for (int ks = 0; ks < NS; ++ks)
        a[ks] = *(const f16x8*)(sK + key * (HD * 2) + (((ks * 4 + g) ^ kswz<HD>(key)) * 16));
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) {
        st[qs][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NS; ++ks) st[qs][kt] = mfma16x16x32(a[ks], qf[qs][ks], st[qs][kt]);
      }
    }
    // online softmax; scores stay unscaled, p = 2^(s*c - m*c) with c = log2(e)/sqrt(hd).
    // Blocks whose every key is visible to every query of the workgroup skip
    // the mask.
    const bool need_mask = kb_cur + KB > seg_n || (own_cur && kb_cur + KB > vis_min);
    f16x8 pb[QS][2];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      float mb = -INFINITY;
      if (need_mask) {
        // key kb + 8g + j is visible iff j < lim - kb - 8g
        const int lim = !own_cur ? seg_n : (seg_n < n_vis[qs] ? seg_n : n_vis[qs]);
        const int dl = lim - kb_cur - 8 * g;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            st[qs][kt][r] = 32 * (kt >> 1) + 4 * (kt & 1) + r < dl ? st[qs][kt][r] : -INFINITY;
      }
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) mb = fmaxf(mb, st[qs][kt][r]);
      mb = max_x32(max_x16(mb));
      // The reference maximum moves only where a score exceeds it by more than
      // 8 / c, so p = 2^(s*c - m*c) stays below 2^8 and the running output is
      // rescaled only on such (rare) blocks.
      const bool grow = mb > m_run[qs] + thr;
      if (__any(grow)) {
        const float m_new = grow ? mb : m_run[qs];
        const float alpha = __builtin_amdgcn_exp2f((m_run[qs] - m_new) * scale_log2);
        l_run[qs] *= alpha;
#pragma unroll
        for (int i = 0; i < NT; ++i) o[qs][i] *= alpha;
        m_run[qs] = m_new;
      }
      const float nmc = -m_run[qs] * scale_log2;
      float ps = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(st[qs][kt][r], scale_log2, nmc));
          ps += e;
          pb[qs][kt >> 1][(kt & 1) * 4 + r] = (f16)e;
        }
      l_run[qs] += ps;
    }
    // O^T += V^T P^T over two 32-key chunks; lane group g's operand is keys
    // 32kc + 8g .. +7 of V^T row `dim`, one 16-byte chunk
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
#pragma unroll
      for (int i = 0; i < NT; ++i) {
        const int dim = 16 * i + c;
        const f16x8 a = *(const f16x8*)(sV + dim * 128 + (((4 * kc + g) ^ vswz(dim)) * 16));
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) o[qs][i] = mfma16x16x32(a, pb[qs][kc], o[qs][i]);
      }
    }
  }

#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const float l_tot = sum_x32(sum_x16(l_run[qs]));
    if (qvalid[qs]) {
      const float inv = 1.0f / l_tot;
      f16* op = (f16*)p.out + (size_t)(row.q_start + tok[qs]) * p.ldo + hq[qs] * HD;
#pragma unroll
      for (int i = 0; i < NT; ++i) {
        f16x4 w = {(f16)(o[qs][i][0] * inv), (f16)(o[qs][i][1] * inv), (f16)(o[qs][i][2] * inv),
                   (f16)(o[qs][i][3] * inv)};
        *(f16x4*)(op + 16 * i + 4 * g) = w;
      }
    }
  }
}

}  // namespace

hipError_t launch_attention(hipStream_t s, const AttnArgs& a) {
  if (a.n_work == 0) return hipSuccess;
  if (a.own_cap > kMaxStoreSlots) return hipErrorInvalidValue;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)a.hd);
  dim3 grid(a.n_work, a.nkv);
  if (a.hd == 128)
    hipLaunchKernelGGL(attn_kernel<128>, grid, dim3(64 * attn_waves<128>()), 0, s, a, scale_log2);
  else if (a.hd == 64)
    hipLaunchKernelGGL(attn_kernel<64>, grid, dim3(64 * attn_waves<64>()), 0, s, a, scale_log2);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace lmop
