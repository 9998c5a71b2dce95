// W4A16 GEMM for gfx950: C = A . deq(W)^T with A fp16 [M][K] (tokens x
// features), W int4 [N][K] with one fp16 scale per 32 input features, fp32
// accumulation on MFMA 16x16x32 f16.  The same body serves FP8 weights (OCP
// E4M3 codes, one fp32 scale per output column: the FP8 checkpoint layout).
// The LM head (fp16 weight) is a kernel of its own at the end of the file.
//
// Tiling.  4 waves side by side along N; a wave owns all (16*MI) tokens of
// the tile and 64 output columns, the workgroup (16*MI) x 256.  K advances
// 64 features (two scale groups) per step through a three-stage LDS ring
// filled by direct global->LDS loads (global_load_lds_dwordx4, 1 KB per wave
// instruction): two steps' tiles stream in while the current step's MFMAs
// run, and one barrier per step suffices.
//   A tile: 128-byte rows, 16-byte chunks XOR-swizzled by row so that one
//           fragment load (16 rows) is free of LDS bank conflicts.
//   int4 tile: copied verbatim from the packed layout (1 KB per 64 columns x
//           32 features: lane 16g+c holds the 8 codes of 4 columns), scales
//           likewise (128 B per 64 columns x 32 features).
// Each wave dequantises its own weight fragments in registers (nibble |
// 0x6400 = 1024 + u in fp16, minus 1032 gives the exact code, times the fp16
// scale: one rounding), once per workgroup, and reuses each for all MI token
// sub-tiles.  Explicit scheduling groups interleave that dequantisation with
// the MFMAs (two VALU per MFMA) so the matrix core is not left idle while a
// wave converts its next fragment.
//
// The MFMA takes the weight fragment as its A operand and the activations
// as its B operand, so the accumulator holds C^T: every lane owns 4
// consecutive output columns of one token, which makes the epilogue's
// stores 8-byte (fp16) or 16-byte (fp32) vectors.
//
// FP8 weights: the tile is 1 KB per 64 columns x 16 features, so a K step
// holds twice the int4 bytes and the ring has two stages (64 KB, two
// workgroups per CU).  A lane's 8 codes convert to fp16 exactly with four
// v_cvt_scalef32_pk_f16_fp8 (every E4M3 value is an fp16 value); the
// per-column scale multiplies the fp32 accumulator before the epilogue.
//
// Workgroups are mapped to tiles XCD-aware: the hardware deals workgroups to
// the 8 XCDs round-robin, so each XCD is given one contiguous range of
// tiles, ordered in groups of GM token tiles so that concurrently running
// tiles on an XCD share A and W panels in that XCD's L2.
#include "common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace lmop {

namespace {

// Dequantises the 8 biased codes of one word (nibble p holds feature 2p for
// p < 4 and 2(p-4)+1 otherwise).  Masking nibbles p and p+4 and or-ing in
// 0x6400 makes fp16 1024 + u, minus 1032 gives the exact code; masking the
// next nibble pair in place makes 1024 + 16u, and one fma by 1/16 with -72
// gives the exact code as well, so one shift by 8 serves all four pairs.
// Times the scale: one rounding.  `mask` and `magic` arrive in registers the
// compiler cannot see through, so (x & mask) | magic becomes one v_and_or.
LMOP_DEVICE f16x8 dequant8(uint32_t w, f16 s, uint32_t mask, uint32_t magic) {
  const f16x2 bias = {(f16)1032.0f, (f16)1032.0f};
  const f16x2 sixteenth = {(f16)0.0625f, (f16)0.0625f};
  const f16x2 bias_hi = {(f16)-72.0f, (f16)-72.0f};
  const f16x2 s2 = {s, s};
  const uint32_t mask_hi = mask << 4;
  const uint32_t w8 = w >> 8;
  const uint32_t t0 = (w & mask) | magic;
  const uint32_t t1 = (w & mask_hi) | magic;
  const uint32_t t2 = (w8 & mask) | magic;
  const uint32_t t3 = (w8 & mask_hi) | magic;
  const f16x2 h0 = (__builtin_bit_cast(f16x2, t0) - bias) * s2;
  const f16x2 h1 = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, t1), sixteenth, bias_hi) * s2;
  const f16x2 h2 = (__builtin_bit_cast(f16x2, t2) - bias) * s2;
  const f16x2 h3 = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, t3), sixteenth, bias_hi) * s2;
  return f16x8{h0.x, h0.y, h1.x, h1.y, h2.x, h2.y, h3.x, h3.y};
}

// The 8 E4M3 codes of two words (feature order, byte 0 first) as fp16,
// exactly: every E4M3 value is an fp16 value, so a unit scale changes nothing.
LMOP_DEVICE f16x8 fp8x8(uint32_t d0, uint32_t d1) {
  const f16x2 a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d0, 1.0f, false);
  const f16x2 b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d0, 1.0f, true);
  const f16x2 c = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d1, 1.0f, false);
  const f16x2 d = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d1, 1.0f, true);
  return f16x8{a.x, a.y, b.x, b.y, c.x, c.y, d.x, d.y};
}

LMOP_DEVICE float silu(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

// 16-byte chunk swizzle of a 128-byte LDS row; with it a fragment load (16
// rows x 4 chunks) is free of bank conflicts on gfx950 (measured with the
// SQ_LDS_BANK_CONFLICT counter)
LMOP_DEVICE int swz(int row) { return row & 7; }

constexpr int BK = 64;
constexpr int BN4 = 256;   // int4 GEMMs: 4 waves x 64 columns
constexpr int GM = 4;      // token tiles per L2 group
constexpr int NSTAGE = 3;  // LDS ring depth

// weight formats of the kernel's weight operand
constexpr int WF_INT4 = 1;  // int4, one fp16 scale per 32 features
constexpr int WF_FP8 = 2;   // OCP E4M3, one fp32 scale per output column

template <int MI, int WF, int NW_ = 4>
struct Cfg {
  // waves per workgroup, side by side along N (64 columns each)
  static constexpr int NW = NW_;
  static constexpr int BN = 64 * NW;
  static constexpr int BM = 16 * MI;
  static constexpr int A_BYTES = BM * 128;
  static constexpr int B_BYTES = WF == WF_INT4 ? BN * 32 : BN * 64;
  static constexpr int S_BYTES = WF == WF_INT4 ? 1024 : 0;
  static constexpr int STAGE = A_BYTES + B_BYTES + S_BYTES;
  static constexpr int NS = WF == WF_FP8 ? 2 : NSTAGE;  // ring stages
  // int4 residual-add tiles prefetch the residual rows into an unread LDS
  // area (1 KB per wave), only so that they are in the caches by the epilogue
  static constexpr int PF = WF == WF_INT4 ? 1024 * NW : 0;
  static constexpr int LDS = NS * STAGE + PF;
  // global->LDS instructions one wave issues per K step (A rows, weight tile, scales)
  static constexpr int A_LOADS = (BM / 8 + NW - 1) / NW;
  static constexpr int B_LOADS = B_BYTES / 1024 / NW;
  static constexpr int LOADS = A_LOADS + B_LOADS + (WF == WF_INT4 ? 1 : 0);
};

// Workgroup: 4 waves side by side along N; wave w owns all BM tokens of the
// tile and columns n0 + 64w .. +63, so every weight fragment is dequantised
// once per workgroup and feeds MI MFMAs.
// 16-token sub-tiles per wave -> workgroups per CU the kernel is built for
template <int MI>
struct Occ {
  static constexpr int value = MI >= 16 ? 1 : 2;
};

template <int MI, int WF, int EPI, int NW_ = 4>
__global__ __launch_bounds__((64 * NW_), Occ<MI>::value) void gemm_kernel(const GemmArgs p) {
  constexpr bool INT4 = WF == WF_INT4;
  using C = Cfg<MI, WF, NW_>;
  constexpr int BM = C::BM, BN = C::BN, NW = C::NW;
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index is uniform; saying so keeps LDS addresses in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c = lane & 15;

  // ---- XCD-aware tile mapping
  const int ntm = (p.M + BM - 1) / BM, ntn = (p.N + BN - 1) / BN;
  const int total = ntm * ntn;
  const int b = blockIdx.x;
  const int xcd = b & 7, j = b >> 3;
  const int per = total >> 3, rem = total & 7;
  const int logical = xcd * per + (xcd < rem ? xcd : rem) + j;
  const int grp = logical / (GM * ntn);
  const int within = logical - grp * GM * ntn;
  const int gsz = (ntm - grp * GM) < GM ? (ntm - grp * GM) : GM;
  const int mt = grp * GM + within % gsz;
  const int nt = within / gsz;
  const int m0 = mt * BM, n0 = nt * BN;

  const int KT = p.K / BK;
  const int KG = p.K / 32;
  const f16* A = (const f16*)p.A;
  // K steps whose stage also prefetches one residual row per wave (the last
  // PFW steps; 4 waves x 32 steps cover the tile's 128 rows)
  const int PFW = KT < BM / NW ? KT : BM / NW;

  // ---- global -> LDS issue of one K step into stage st; every wave issues
  // exactly C::LOADS instructions, which the vmcnt waits below rely on.
  // Each load is a base in scalar registers (moved by kt) plus a per-lane
  // 32-bit byte offset computed once, and an LDS destination in a scalar
  // register.
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_ptr_t)smem;
  uint32_t aoff[C::A_LOADS];
#pragma unroll
  for (int i = 0; i < C::A_LOADS; ++i) {
    int q = wave + NW * i;  // 8 rows per instruction
    if (q >= BM / 8) q = BM / 8 - 1;  // surplus waves repeat the last rows
    const int r = q * 8 + (lane >> 3);
    const int chunk = (lane & 7) ^ swz(r);
    const int gm = m0 + r < p.M ? r : p.M - 1 - m0;  // row within the tile, clamped
    aoff[i] = (uint32_t)(gm * p.lda + chunk * 8) * 2u;
  }
  const char* abase = (const char*)(A + (size_t)m0 * p.lda);
  const size_t nb0 = (size_t)(n0 >> 6);
  // int4 scales: lane group pi = lane / 8 fetches pair pi's 128 bytes
  const uint32_t soff = (uint32_t)(((lane >> 4) * KG + ((lane >> 3) & 1)) * 128 + (lane & 7) * 16);
  auto issue = [&](int st, int kt) {
    const uint32_t sA = lds0 + (uint32_t)(st * C::STAGE);
    const uint32_t sB = sA + C::A_BYTES;
    const uint32_t sS = sB + C::B_BYTES;
#pragma unroll
    for (int i = 0; i < C::A_LOADS; ++i) {
      int q = wave + NW * i;
      if (q >= BM / 8) q = BM / 8 - 1;
      g2l16_m0(abase + kt * BK * 2, aoff[i], sA + (uint32_t)q * 1024u);
    }
    if constexpr (INT4) {
#pragma unroll
      for (int i = 0; i < C::B_LOADS; ++i) {  // (64-column block, group) pairs
        const int q = wave + NW * i;
        const char* b = (const char*)p.bq + ((nb0 + (q >> 1)) * KG + kt * 2 + (q & 1)) * 1024;
        g2l16_m0(b, (uint32_t)lane * 16u, sB + (uint32_t)q * 1024u);
      }
      {  // scales: 8 pairs x 128 B = one 1 KB instruction, spread over the waves
        const char* b = (const char*)p.bs + (nb0 * KG + kt * 2) * 128;
        if ((lane >> 4) == wave) g2l16_m0(b, soff, sS);
      }
      if constexpr (EPI == EPI_ADD_F32) {
        // the residual row r of the tile (1 KB: this wave's 256 columns),
        // issued after the stage so the waits below can count it
        if (kt >= KT - PFW) {
          const int r = (kt - (KT - PFW)) * NW + wave;
          int gm = m0 + (r < BM ? r : BM - 1);
          gm = gm < p.M ? gm : p.M - 1;
          int col = n0 + lane * 4;
          col = col + 4 <= p.n_out ? col : p.n_out - 4;
          g2l16_m0((const char*)(p.X + (size_t)gm * p.ldx), (uint32_t)col * 4u,
                   lds0 + (uint32_t)(C::NS * C::STAGE + wave * 1024));
        }
      }
    } else if constexpr (WF == WF_FP8) {
      // 1 KB chunks: (64-column block, group) pair q >> 1, half q & 1
#pragma unroll
      for (int i = 0; i < C::B_LOADS; ++i) {
        const int q = wave + NW * i;
        const int pr = q >> 1;
        const size_t blk = (nb0 + (pr >> 1)) * KG + kt * 2 + (pr & 1);
        g2l16_m0((const char*)p.bq + (blk * 2 + (q & 1)) * 1024, (uint32_t)lane * 16u,
                 sB + (uint32_t)q * 1024u);
      }
    }
  };

  // dequant constants kept opaque to the optimiser (see dequant8)
  uint32_t dq_mask = 0x000F000Fu, dq_magic = 0x64006400u;
  asm volatile("" : "+s"(dq_mask));
  asm volatile("" : "+v"(dq_magic));

  f32x4 acc[4][MI];
#pragma unroll
  for (int f = 0; f < 4; ++f)
#pragma unroll
    for (int i = 0; i < MI; ++i) acc[f][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  if constexpr (INT4) {
    issue(0, 0);
    if (KT > 1) issue(1, 1);
    for (int kt = 0; kt < KT; ++kt) {
      // this step's stage is complete once at most the next step's loads
      // (and the residual prefetch issued after them) are in flight
      if (kt + 1 < KT) {
        if (EPI == EPI_ADD_F32 && kt + 1 >= KT - PFW)
          wait_vmcnt<C::LOADS + 1>();
        else
          wait_vmcnt<C::LOADS>();
      } else {
        wait_vmcnt<0>();
      }
      barrier();
      if (kt + 2 < KT) issue((kt + 2) % NSTAGE, kt + 2);
      const char* sA = smem + (kt % NSTAGE) * C::STAGE;
      const char* sB = sA + C::A_BYTES;
      const char* sS = sB + C::B_BYTES;
        // both 32-feature groups' activation fragments, codes and scales are
        // read up front; then one weight fragment at a time
        f16x8 a[2][MI];
        uint4 codes[2];
        f16x4 s4[2];
  #pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
  #pragma unroll
          for (int i = 0; i < MI; ++i) {
            const int r = 16 * i + c;
            a[kk][i] = *(const f16x8*)(sA + r * 128 + (((kk * 4 + g) ^ swz(r)) * 16));
          }
          const int q = wave * 2 + kk;
          codes[kk] = *(const uint4*)(sB + q * 1024 + lane * 16);
          s4[kk] = *(const f16x4*)(sS + q * 128 + c * 8);
        }
  #pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
  #pragma unroll
          for (int f = 0; f < 4; ++f) {
            const uint32_t cw = f == 0 ? codes[kk].x : f == 1 ? codes[kk].y : f == 2 ? codes[kk].z : codes[kk].w;
            const f16x8 w = dequant8(cw, s4[kk][f], dq_mask, dq_magic);
  #pragma unroll
            for (int i = 0; i < MI; ++i) acc[f][i] = mfma16x16x32(w, a[kk][i], acc[f][i]);
          }
        }
        // Schedule: the LDS reads first, then the first fragment's dequant (13
        // VALU), then every MFMA followed by up to two VALU, so the remaining
        // dequant work issues while earlier MFMAs run instead of in VALU-only
        // stretches that leave the matrix core idle.
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * MI + 4, 0);  // DS reads
        __builtin_amdgcn_sched_group_barrier(0x002, 13, 0);          // VALU
  #pragma unroll
        for (int j = 0; j < 8 * MI; ++j) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // VALU
        }
    }
  } else if constexpr (WF == WF_FP8) {
    // two stages: the next step's tiles load while this step's MFMAs run
    issue(0, 0);
    for (int kt = 0; kt < KT; ++kt) {
      // this step's loads are the only ones in flight
      wait_vmcnt<0>();
      barrier();
      if (kt + 1 < KT) issue((kt + 1) & 1, kt + 1);
      const char* sA = smem + (kt & 1) * C::STAGE;
      const char* sB = sA + C::A_BYTES;
      f16x8 a[2][MI];
      uint4 cw[2][2];  // [group][half]: half h holds columns 16*(2h + f') + c
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
        for (int i = 0; i < MI; ++i) {
          const int r = 16 * i + c;
          a[kk][i] = *(const f16x8*)(sA + r * 128 + (((kk * 4 + g) ^ swz(r)) * 16));
        }
        const int q = wave * 2 + kk;
        cw[kk][0] = *(const uint4*)(sB + q * 2048 + lane * 16);
        cw[kk][1] = *(const uint4*)(sB + q * 2048 + 1024 + lane * 16);
      }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          const uint4 h = cw[kk][f >> 1];
          const f16x8 w = (f & 1) ? fp8x8(h.z, h.w) : fp8x8(h.x, h.y);
#pragma unroll
          for (int i = 0; i < MI; ++i) acc[f][i] = mfma16x16x32(w, a[kk][i], acc[f][i]);
        }
      }
      __builtin_amdgcn_sched_group_barrier(0x100, 2 * MI + 4, 0);  // DS reads
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);           // VALU
#pragma unroll
      for (int j = 0; j < 8 * MI; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);  // VALU
      }
    }
  }

  // ------------------------------------------------------------ epilogue
  // acc[f][i][r] = C[m][n], m = m0 + 16i + c, n = n0 + 64*wave + 16f + 4g + r
  const int mrow = m0 + c;
  const int ncol = n0 + wave * 64 + 4 * g;
  if constexpr (WF == WF_FP8) {
    // the FP8 weight's per-column scale
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const float4 sc = *(const float4*)(p.bsc + ncol + 16 * f);
#pragma unroll
      for (int i = 0; i < MI; ++i) acc[f][i] = acc[f][i] * f32x4{sc.x, sc.y, sc.z, sc.w};
    }
  }
  if constexpr (EPI == EPI_STORE_F16) {
    f16* Cp = (f16*)p.C;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const int m = mrow + 16 * i;
      if (m >= p.M) continue;
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const int n = ncol + 16 * f;
        if (n < p.n_out) {
          const f32x4 v = acc[f][i];
          *(f16x4*)(Cp + (size_t)m * p.ldc + n) = f16x4{(f16)v[0], (f16)v[1], (f16)v[2], (f16)v[3]};
        }
      }
    }
  } else if constexpr (EPI == EPI_ADD_F32) {
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const int m = mrow + 16 * i;
      if (m >= p.M) continue;
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const int n = ncol + 16 * f;
        if (n < p.n_out) {
          float4* xp = (float4*)(p.X + (size_t)m * p.ldx + n);
          float4 x = *xp;
          const f32x4 v = acc[f][i];
          x.x += v[0];
          x.y += v[1];
          x.z += v[2];
          x.w += v[3];
          *xp = x;
        }
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // the wave's 64-column block holds gate columns blk*32 + 0..31 (sub-tiles
    // 0, 1) and the matching up columns (sub-tiles 2, 3)
    f16* Cp = (f16*)p.C;
    const int blk = (n0 >> 6) + wave;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const int m = mrow + 16 * i;
      if (m >= p.M) continue;
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        const int col = blk * 32 + 16 * f + 4 * g;
        if (col < p.n_out) {
          const f32x4 gt = acc[f][i], up = acc[f + 2][i];
          *(f16x4*)(Cp + (size_t)m * p.ldc + col) =
              f16x4{(f16)(silu(gt[0]) * up[0]), (f16)(silu(gt[1]) * up[1]),
                    (f16)(silu(gt[2]) * up[2]), (f16)(silu(gt[3]) * up[3])};
        }
      }
    }
  } else if constexpr (EPI == EPI_QKV) {
    const int blk = (n0 >> 6) + wave;
    const int bph = p.hd >> 6;  // 64-column blocks per head
    const int nqb = p.nq * bph, nkb = p.nkv * bph;
    if (blk < nqb + 2 * nkb) {
      const int sec = blk < nqb ? 0 : (blk < nqb + nkb ? 1 : 2);
      const int hb = blk - (sec == 0 ? 0 : (sec == 1 ? nqb : nqb + nkb));
      const int head = hb / bph, sub = hb - head * bph;
      const int half = p.hd >> 1;
      const int kvdim = p.nkv * p.hd;
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int m = mrow + 16 * i;
        if (m >= p.M) continue;
        const int sl = p.slot[m];
        if (sec < 2) {
          const float2* cs = p.rope + (size_t)p.pos[m] * half;
          f16* dst = sec == 0 ? (f16*)p.qout + (size_t)m * p.nq * p.hd + head * p.hd
                              : (f16*)p.kc + (size_t)sl * kvdim + head * p.hd;
#pragma unroll
          for (int f = 0; f < 2; ++f) {
            const int d = 32 * sub + 16 * f + 4 * g;
            const f32x4 x1 = acc[f][i], x2 = acc[f + 2][i];
            const float4 c01 = *(const float4*)(cs + d);
            const float4 c23 = *(const float4*)(cs + d + 2);
            const float cr[4] = {c01.x, c01.z, c23.x, c23.z};
            const float sr[4] = {c01.y, c01.w, c23.y, c23.w};
            f16x4 y1, y2;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              y1[r] = (f16)(x1[r] * cr[r] - x2[r] * sr[r]);
              y2[r] = (f16)(x1[r] * sr[r] + x2[r] * cr[r]);
            }
            *(f16x4*)(dst + d) = y1;
            *(f16x4*)(dst + half + d) = y2;
          }
        } else {
          f16* vt = (f16*)p.vt + (size_t)head * p.hd * p.cap + sl;
#pragma unroll
          for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              vt[(size_t)(64 * sub + 16 * f + 4 * g + r) * p.cap] = (f16)acc[f][i][r];
        }
      }
    }
  }
}

template <int MI, int WF, int EPI, int NW = 4>
hipError_t launch_cfg(hipStream_t s, const GemmArgs& a) {
  using C = Cfg<MI, WF, NW>;
  const int tiles = ((a.M + C::BM - 1) / C::BM) * ((a.N + C::BN - 1) / C::BN);
  if (tiles == 0) return hipSuccess;
  // set once per instantiation (a function-local static is initialised once,
  // also when several threads launch)
  static const hipError_t attr = hipFuncSetAttribute(
      (const void*)gemm_kernel<MI, WF, EPI, NW>, hipFuncAttributeMaxDynamicSharedMemorySize,
      C::LDS);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((gemm_kernel<MI, WF, EPI, NW>), dim3(tiles), dim3(64 * NW), C::LDS, s, a);
  return hipGetLastError();
}

template <int WF, int EPI>
hipError_t launch_epi(hipStream_t s, const GemmArgs& a) {
  // the largest token tile that still gives every CU a workgroup
  const long ntn = a.N / 256;
  if ((long)((a.M + 127) / 128) * ntn >= 256) return launch_cfg<8, WF, EPI>(s, a);
  if ((long)((a.M + 63) / 64) * ntn >= 256) return launch_cfg<4, WF, EPI>(s, a);
  return launch_cfg<2, WF, EPI>(s, a);
}

// ---------------------------------------------------------------- LM head
// 16-byte chunk swizzle of a 64-byte LDS row: the 8 lanes a ds_read_b128
// serves together (rows c .. c+7 of a fragment, one chunk) fall on 8
// distinct 16-byte bank groups of a 128-byte window
LMOP_DEVICE int swz64(int row) { return (row >> 1) & 3; }

// ---------------------------------------------------------------- LM head
// z = W_lm . h for R token rows: the head weight W_lm fp16 (tiled, see
// kHeadTileRows) is the vocabulary operand (M), the final-normalised rows h
// fp16 [R][K] the token operand (N); both stream through an LDS ring by
// direct global->LDS loads, 32 features per step in 64-byte LDS rows.  A
// workgroup of 8 waves holds two vocabulary tiles (256 rows) and 64*F token
// rows: wave w computes vocabulary tile w / 4 of the pair for token-row
// group w % 4 (16*F rows).  The two tiles share the token rows in LDS, so
// token rows cross from L2 once per 256 vocabulary rows, and one workgroup
// per CU affords a ring of NS stages (four: three steps of loads in flight).
// Per token and 128-entry vocabulary chunk the epilogue writes (max, sum
// exp) and the allowed tokens' logits; the chunking never depends on the
// tile or the number of rows, so a row's log-probabilities do not depend on
// how rows are batched.  (One 128-row vocabulary tile per 4-wave workgroup,
// two workgroups per CU, ran 12-14% longer; token rows loaded straight into
// registers ran ~35% longer than through the ring.)
template <int F_, int NS_>
struct Head2Cfg {
  static constexpr int F = F_, NS = NS_, NW = 8, BK = 32, MI = 8;
  static constexpr int BM = 2 * kHeadTileRows, BN = 4 * 16 * F;
  static constexpr int A_BYTES = BM * 64, T_BYTES = BN * 64;
  static constexpr int STAGE = A_BYTES + T_BYTES;
  static constexpr int LDS = NS * STAGE;
  static_assert(NS >= 2 && LDS <= 160 * 1024, "LDS of one CU");
  static constexpr int T_BLOCKS = BN / 16;
  static constexpr int T_MAX = (T_BLOCKS + NW - 1) / NW;  // token blocks of the first waves
  static constexpr int T_FULL = T_BLOCKS % NW == 0 ? NW : T_BLOCKS % NW;  // waves with T_MAX
  static constexpr int LOADS_HI = 2 + T_MAX, LOADS_LO = 2 + T_MAX - 1;
  static_assert((NS - 2) * LOADS_HI <= 63, "loads in flight fit the vmcnt counter");
};

template <int F, int NS_>
__global__ __launch_bounds__(512, 1) void head2_kernel(const GemmArgs p) {
  using C = Head2Cfg<F, NS_>;
  constexpr int BK = C::BK, BM = C::BM, BN = C::BN, NS = C::NS, MI = C::MI;
  constexpr int A_BYTES = C::A_BYTES, STAGE = C::STAGE;
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c = lane & 15;
  const int half = wave >> 2, grp_t = wave & 3;

  // XCD-aware tile order as in gemm_kernel
  const int ntm = (p.M + BM - 1) / BM, ntn = (p.N + BN - 1) / BN;
  const int total = ntm * ntn;
  const int b = blockIdx.x;
  const int xcd = b & 7, j = b >> 3;
  const int per = total >> 3, rem = total & 7;
  const int logical = xcd * per + (xcd < rem ? xcd : rem) + j;
  const int grp = logical / (GM * ntn);
  const int within = logical - grp * GM * ntn;
  const int gsz = (ntm - grp * GM) < GM ? (ntm - grp * GM) : GM;
  const int mt = grp * GM + within % gsz;
  const int nt = within / gsz;
  const int n0 = nt * BN;
  const int w0 = n0 + grp_t * 16 * F;  // this wave's first token row
  const int KT = p.K / BK;
  const int n_tiles = (p.M + kHeadTileRows - 1) / kHeadTileRows;
  const f16* W = (const f16*)p.A;
  const f16* H = (const f16*)p.bh;

  // loads: wave w fetches 16-row block w of both vocabulary tiles (the
  // second clamped to the last tile of the weight) and token blocks w, w+8,
  // ...; the first T_FULL waves have one token block more, so the waits
  // take one of two compile-time counts
  const int rr = lane >> 2, pc = lane & 3;
  const int ra = wave * 16 + rr;
  const uint32_t aoff = (uint32_t)(ra * 64 + (pc ^ swz64(ra)) * 16);
  const char* wbase[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int t = 2 * mt + h < n_tiles ? 2 * mt + h : n_tiles - 1;
    wbase[h] = (const char*)(W + (size_t)t * KT * (kHeadTileRows * 32));
  }
  uint32_t toff[C::T_MAX];
#pragma unroll
  for (int i = 0; i < C::T_MAX; ++i) {
    int q = wave + 8 * i;
    if (q >= C::T_BLOCKS) q = C::T_BLOCKS - 1;
    const int r = q * 16 + rr;
    const int gn = n0 + r < p.N ? r : p.N - 1 - n0;
    toff[i] = (uint32_t)(gn * p.ldb + (pc ^ swz64(r)) * 8) * 2u;
  }
  const char* hbase = (const char*)(H + (size_t)n0 * p.ldb);
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_ptr_t)smem;
  const bool t_hi = wave < C::T_FULL;
  auto issue = [&](int st, int kt) {
    const uint32_t sA = lds0 + (uint32_t)(st * STAGE);
    const uint32_t sT = sA + A_BYTES;
#pragma unroll
    for (int h = 0; h < 2; ++h)
      g2l16_m0(wbase[h] + (size_t)kt * (kHeadTileRows * 64), aoff,
               sA + (uint32_t)(h * kHeadTileRows * 64 + wave * 1024));
#pragma unroll
    for (int i = 0; i < C::T_MAX; ++i)
      if (i < C::T_MAX - 1 || t_hi)
        g2l16_m0(hbase + kt * BK * 2, toff[i], sT + (uint32_t)(wave + 8 * i) * 1024u);
  };

  f32x4 acc[F][MI];
#pragma unroll
  for (int f = 0; f < F; ++f)
#pragma unroll
    for (int i = 0; i < MI; ++i) acc[f][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  const bool wave_active = w0 < p.N;
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < KT) issue(st, st);
  for (int kt = 0; kt < KT; ++kt) {
    // this step's stage is complete once at most the later steps' loads
    // (NS - 2 stages of them) are in flight; near the end, none
    if (kt + NS - 2 < KT) {
      if (t_hi)
        wait_vmcnt<(NS - 2) * C::LOADS_HI>();
      else
        wait_vmcnt<(NS - 2) * C::LOADS_LO>();
    } else {
      wait_vmcnt<0>();
    }
    barrier();
    if (kt + NS - 1 < KT) issue((kt + NS - 1) % NS, kt + NS - 1);
    if (wave_active) {
      const char* sA = smem + (kt % NS) * STAGE + half * (kHeadTileRows * 64);
      const char* sT = smem + (kt % NS) * STAGE + A_BYTES;
      f16x8 a[MI], t[F];
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int r = 16 * i + c;
        a[i] = *(const f16x8*)(sA + r * 64 + ((g ^ swz64(r)) * 16));
      }
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const int r = grp_t * 16 * F + 16 * f + c;
        t[f] = *(const f16x8*)(sT + r * 64 + ((g ^ swz64(r)) * 16));
      }
#pragma unroll
      for (int f = 0; f < F; ++f)
#pragma unroll
        for (int i = 0; i < MI; ++i) acc[f][i] = mfma16x16x32(t[f], a[i], acc[f][i]);
    }
  }

  // acc[f][i][r] = z[vocabulary m0 + 16i + c][token w0 + 16f + 4g + r]
  const int chunk = 2 * mt + half;
  const int n_chunks = n_tiles;
  if (chunk >= n_chunks) return;  // a pair's second tile past the vocabulary
  const int mrow = chunk * kHeadTileRows + c;
  const int ncol = w0 + 4 * g;
#pragma unroll
  for (int f = 0; f < F; ++f)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int n = ncol + 16 * f + r;  // token
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < MI; ++i)
        if (mrow + 16 * i < p.M) mx = fmaxf(mx, acc[f][i][r]);
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, shfl_xor(mx, o));
      float sm = 0.f;
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int v = mrow + 16 * i;  // vocabulary entry
        if (v < p.M) {
          const float z = acc[f][i][r];
          sm += __expf(z - mx);
          if (n < p.N) {
            const int si = p.sel[v];
            if (si >= 0) p.zsel[(size_t)n * p.n_sel + si] = z;
            if (p.dump) p.dump[(size_t)n * p.ld_dump + v] = z;
          }
        }
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) sm += shfl_xor(sm, o);
      if (c == 0 && n < p.N) p.part[(size_t)n * n_chunks + chunk] = make_float2(mx, sm);
    }
}

template <int F, int NS>
hipError_t launch_head2(hipStream_t s, const GemmArgs& a) {
  using C = Head2Cfg<F, NS>;
  const int tiles = ((a.M + C::BM - 1) / C::BM) * ((a.N + C::BN - 1) / C::BN);
  if (tiles == 0) return hipSuccess;
  static const hipError_t attr = hipFuncSetAttribute(
      (const void*)head2_kernel<F, NS>, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((head2_kernel<F, NS>), dim3(tiles), dim3(512), C::LDS, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_f16(hipStream_t s, const GemmArgs& a, int epi) {
  using H256 = Head2Cfg<4, 4>;  // 256-token tile
  using H320 = Head2Cfg<5, 4>;  // 320-token tile
  static_assert(kHeadTileRows == kHeadVocabChunk, "partials per vocabulary chunk");
  if (a.K % 32 != 0 || epi != EPI_HEAD || a.ldb % 8 != 0)
    return hipErrorInvalidValue;
  // per-lane token-row offsets are 32-bit byte offsets within one tile's rows
  if ((size_t)512 * a.ldb * 2 >= (size_t(1) << 31)) return hipErrorInvalidValue;
  // A workgroup's time barely depends on how many of its token rows are
  // real, so the tile that needs fewer token tiles wins; a full 320-token
  // tile runs about 10% longer than a full 256-token one.  Each logit's
  // accumulation order is the same in both, so the choice never changes a bit.
  const int t256 = (a.N + H256::BN - 1) / H256::BN, t320 = (a.N + H320::BN - 1) / H320::BN;
  if (10 * t256 > 11 * t320) return launch_head2<5, 4>(s, a);
  return launch_head2<4, 4>(s, a);
}

hipError_t launch_gemm_w4(hipStream_t s, const GemmArgs& a, int epi) {
  // the packed weight is padded to 256 columns so every tile shape divides it
  if (a.K % BK != 0 || a.N % 256 != 0) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_STORE_F16: return launch_epi<WF_INT4, EPI_STORE_F16>(s, a);
    case EPI_ADD_F32: return launch_epi<WF_INT4, EPI_ADD_F32>(s, a);
    case EPI_SWIGLU: return launch_epi<WF_INT4, EPI_SWIGLU>(s, a);
    case EPI_QKV: return launch_epi<WF_INT4, EPI_QKV>(s, a);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_w8(hipStream_t s, const GemmArgs& a, int epi) {
  // the packed weight is padded to 256 columns (and its scales with it)
  if (a.K % BK != 0 || a.N % 256 != 0 || !a.bsc) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_STORE_F16: return launch_epi<WF_FP8, EPI_STORE_F16>(s, a);
    case EPI_ADD_F32: return launch_epi<WF_FP8, EPI_ADD_F32>(s, a);
    case EPI_SWIGLU: return launch_epi<WF_FP8, EPI_SWIGLU>(s, a);
    case EPI_QKV: return launch_epi<WF_FP8, EPI_QKV>(s, a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace lmop
