// W4A16 GEMM for gfx950: C = A . deq(W)^T with A fp16 [M][K], W int4 with one
// fp16 scale per 32 input features, fp32 accumulation on MFMA 16x16x32 f16.
//
// Workgroup: 256 threads = 4 waves in a 2 (M) x 2 (N) grid; wave tile
// (16*MI) x 64, workgroup tile (32*MI) x 128, K step 64 (two scale groups).
// The A tile goes global -> registers -> LDS (padded rows); the next tile's
// loads are issued before the current tile's MFMAs.  Each wave fetches its
// own int4 weight words straight from global memory (the packed layout puts
// one 16-byte word per lane per group, so a wave reads 1 KB contiguously),
// dequantises them in registers (nibble | 0x6400 -> 1024 + u, minus 1032,
// times the scale: exact code, one fp16 rounding of code * scale) and reuses
// each dequantised fragment for all MI row sub-tiles.
//
// The same kernel body, with an fp16 weight, computes the LM head; its
// epilogue reduces every 64-column slice of logits to (max, sum exp) and
// extracts the logits of the allowed tokens, so no [rows x vocab] matrix is
// written unless a debug dump is requested.
#include "common.h"
#include "kernels.h"

namespace lmop {

namespace {

LMOP_DEVICE f16x8 dequant8(uint32_t w, f16 s) {
  const uint32_t kMask = 0x000F000Fu, kMagic = 0x64006400u;
  const f16x2 bias = {(f16)1032.0f, (f16)1032.0f};
  const f16x2 s2 = {s, s};
  f16x2 h0 = (__builtin_bit_cast(f16x2, (w & kMask) | kMagic) - bias) * s2;
  f16x2 h1 = (__builtin_bit_cast(f16x2, ((w >> 4) & kMask) | kMagic) - bias) * s2;
  f16x2 h2 = (__builtin_bit_cast(f16x2, ((w >> 8) & kMask) | kMagic) - bias) * s2;
  f16x2 h3 = (__builtin_bit_cast(f16x2, ((w >> 12) & kMask) | kMagic) - bias) * s2;
  return f16x8{h0.x, h0.y, h1.x, h1.y, h2.x, h2.y, h3.x, h3.y};
}

LMOP_DEVICE float silu(float g) { return g / (1.0f + __expf(-g)); }

constexpr int BN = 128;
constexpr int BK = 64;
constexpr int LDS_ROW = BK + 8;  // halves; padding spreads rows over LDS banks

template <int MI, bool INT4, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmArgs p) {
  constexpr int BM = 32 * MI;
  constexpr int ACH = BM * (BK / 8) / 256;  // 16-byte A chunks per thread per K step
  __shared__ f16 sA[BM * LDS_ROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int g = lane >> 4, c = lane & 15;
  const int ntn = (p.N + BN - 1) / BN;
  const int mt = blockIdx.x / ntn, nt = blockIdx.x - mt * ntn;
  const int m0 = mt * BM, n0 = nt * BN;
  const int KT = p.K / BK;
  const int KG = p.K / 32;
  const f16* A = (const f16*)p.A;

  f32x4 acc[MI][4];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int f = 0; f < 4; ++f) acc[i][f] = f32x4{0.f, 0.f, 0.f, 0.f};

  f16x8 areg[ACH];
  auto loadA = [&](int kt) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int ch = tid + i * 256, r = ch >> 3, cc = (ch & 7) * 8;
      const int gm = m0 + r;
      if (gm < p.M)
        areg[i] = *(const f16x8*)(A + (size_t)gm * p.lda + kt * BK + cc);
      else
        areg[i] = f16x8{0, 0, 0, 0, 0, 0, 0, 0};
    }
  };
  auto storeA = [&]() {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int ch = tid + i * 256, r = ch >> 3, cc = (ch & 7) * 8;
      *(f16x8*)(sA + r * LDS_ROW + cc) = areg[i];
    }
  };

  // weight fragments of one K step (two groups)
  uint4 bq[2];
  uint2 bsc[2];
  f16x8 bh[2][4];
  const int nb = (n0 >> 6) + wn;  // global 64-column block of this wave
  auto loadB = [&](int kt) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int kg = kt * 2 + j;
      if constexpr (INT4) {
        const size_t blk = (size_t)nb * KG + kg;
        bq[j] = ((const uint4*)p.bq)[blk * 64 + lane];
        bsc[j] = ((const uint2*)p.bs)[blk * 16 + c];
      } else {
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          int n = n0 + wn * 64 + f * 16 + c;
          n = n < p.N ? n : p.N - 1;  // clamped; masked in the epilogue
          bh[j][f] = *(const f16x8*)((const f16*)p.bh + (size_t)n * p.ldb + kg * 32 + g * 8);
        }
      }
    }
  };

  loadA(0);
  loadB(0);
  for (int kt = 0; kt < KT; ++kt) {
    __syncthreads();
    storeA();
    __syncthreads();
    uint4 cq[2] = {bq[0], bq[1]};
    uint2 cs[2] = {bsc[0], bsc[1]};
    f16x8 ch[2][4];
    if constexpr (!INT4) {
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int f = 0; f < 4; ++f) ch[j][f] = bh[j][f];
    }
    if (kt + 1 < KT) {
      loadA(kt + 1);
      loadB(kt + 1);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      f16x8 b[4];
      if constexpr (INT4) {
        const f16x4 s4 = __builtin_bit_cast(f16x4, cs[j]);
        b[0] = dequant8(cq[j].x, s4.x);
        b[1] = dequant8(cq[j].y, s4.y);
        b[2] = dequant8(cq[j].z, s4.z);
        b[3] = dequant8(cq[j].w, s4.w);
      } else {
#pragma unroll
        for (int f = 0; f < 4; ++f) b[f] = ch[j][f];
      }
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const f16x8 a =
            *(const f16x8*)(sA + (wm * 16 * MI + 16 * i + c) * LDS_ROW + j * 32 + g * 8);
#pragma unroll
        for (int f = 0; f < 4; ++f) acc[i][f] = mfma16x16x32(a, b[f], acc[i][f]);
      }
    }
  }

  // ------------------------------------------------------------ epilogue
  const int row_base = m0 + wm * 16 * MI + 4 * g;
  if constexpr (EPI == EPI_STORE_F16) {
    f16* C = (f16*)p.C;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const int col = n0 + wn * 64 + 16 * f + c;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = row_base + 16 * i + r;
          if (row < p.M && col < p.n_out) C[(size_t)row * p.ldc + col] = (f16)acc[i][f][r];
        }
      }
  } else if constexpr (EPI == EPI_ADD_F32) {
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const int col = n0 + wn * 64 + 16 * f + c;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = row_base + 16 * i + r;
          if (row < p.M && col < p.n_out) p.X[(size_t)row * p.ldx + col] += acc[i][f][r];
        }
      }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // block nb holds gate columns nb*32 + 0..31 in f = 0,1 and the matching up
    // columns in f = 2,3
    f16* C = (f16*)p.C;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        const int col = nb * 32 + 16 * f + c;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = row_base + 16 * i + r;
          if (row < p.M && col < p.n_out)
            C[(size_t)row * p.ldc + col] = (f16)(silu(acc[i][f][r]) * acc[i][f + 2][r]);
        }
      }
  } else {  // EPI_HEAD
    const int n_chunks = (p.N + 63) / 64;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = row_base + 16 * i + r;
        float mx = -INFINITY;
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          const int col = n0 + wn * 64 + 16 * f + c;
          if (col < p.N) mx = fmaxf(mx, acc[i][f][r]);
        }
        // lanes 16g .. 16g+15 hold the 64 columns of this row
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, shfl_xor(mx, o));
        float sm = 0.f;
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          const int col = n0 + wn * 64 + 16 * f + c;
          if (col < p.N) {
            const float z = acc[i][f][r];
            sm += __expf(z - mx);
            if (row < p.M) {
              const int si = p.sel[col];
              if (si >= 0) p.zsel[(size_t)row * p.n_sel + si] = z;
              if (p.dump) p.dump[(size_t)row * p.ld_dump + col] = z;
            }
          }
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) sm += shfl_xor(sm, o);
        if (c == 0 && row < p.M && nb < n_chunks)
          p.part[(size_t)row * n_chunks + nb] = make_float2(mx, sm);
      }
    }
  }
}

template <int MI, bool INT4, int EPI>
hipError_t launch_mi(hipStream_t s, const GemmArgs& a) {
  constexpr int BM = 32 * MI;
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<MI, INT4, EPI>), dim3(tiles), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <bool INT4, int EPI>
hipError_t launch_epi(hipStream_t s, const GemmArgs& a) {
  if (a.M > 1024) return launch_mi<8, INT4, EPI>(s, a);
  if (a.M > 256) return launch_mi<4, INT4, EPI>(s, a);
  return launch_mi<2, INT4, EPI>(s, a);
}

}  // namespace

hipError_t launch_gemm_w4(hipStream_t s, const GemmArgs& a, int epi) {
  if (a.K % BK != 0 || a.N % BN != 0) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_STORE_F16: return launch_epi<true, EPI_STORE_F16>(s, a);
    case EPI_ADD_F32: return launch_epi<true, EPI_ADD_F32>(s, a);
    case EPI_SWIGLU: return launch_epi<true, EPI_SWIGLU>(s, a);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_f16(hipStream_t s, const GemmArgs& a, int epi) {
  if (a.K % BK != 0 || epi != EPI_HEAD || a.ldb % 8 != 0) return hipErrorInvalidValue;
  return launch_epi<false, EPI_HEAD>(s, a);
}

}  // namespace lmop
