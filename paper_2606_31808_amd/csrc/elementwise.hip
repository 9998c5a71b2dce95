// HBM-bound kernels of the row-evaluation path: embedding gather, RMSNorm
// (fp32 residual -> fp16 GEMM operand), the load-time int4 repack, and the
// per-row finish of the constrained LM head.  (RoPE and the key/value write
// live in the QKV GEMM's epilogue.)
#include "common.h"
#include "kernels.h"

namespace lmop {

namespace {

// --------------------------------------------------------------- fill
// p[i] = value for i < n 32-bit words (clears scratch and KV stores with a
// kernel, so no memset node lands in a caller's captured graph)
__global__ __launch_bounds__(256) void fill_u32_kernel(uint32_t* __restrict__ p, size_t n,
                                                       uint32_t value) {
  const size_t stride = (size_t)gridDim.x * 256 * 4;
  for (size_t i = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4; i < n; i += stride) {
    if (i + 4 <= n) {
      *(uint4*)(p + i) = make_uint4(value, value, value, value);
    } else {
      for (size_t j = i; j < n; ++j) p[j] = value;
    }
  }
}

// --------------------------------------------------------------- embedding
// x[t][:] = fp32(E[tok[t]][:]); one workgroup per token, 8 halves per thread-iteration
__global__ __launch_bounds__(256) void embed_kernel(const int32_t* __restrict__ tok,
                                                    const f16* __restrict__ emb, int d,
                                                    float* __restrict__ x) {
  const int t = blockIdx.x;
  const f16* src = emb + (size_t)tok[t] * d;
  float* dst = x + (size_t)t * d;
  for (int j = threadIdx.x * 8; j < d; j += 256 * 8) {
    const f16x8 v = *(const f16x8*)(src + j);
    float4 lo = make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
    float4 hi = make_float4((float)v[4], (float)v[5], (float)v[6], (float)v[7]);
    *(float4*)(dst + j) = lo;
    *(float4*)(dst + j + 4) = hi;
  }
}

// --------------------------------------------------------------- RMSNorm
// out[i] = fp16(x_i / sqrt(mean(x_i^2) + eps) * gamma); one workgroup per row.
// The sum of squares is reduced in a fixed order, so a row's result does not
// depend on which other rows share the launch.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ x, int ldx,
                                                      const float* const* __restrict__ rowptr,
                                                      const float* __restrict__ gamma, int d,
                                                      float eps, f16* __restrict__ out, int ldo) {
  const int i = blockIdx.x;
  const float* row = rowptr ? rowptr[i] : x + (size_t)i * ldx;
  __shared__ float red[4];
  float ss = 0.f;
  for (int j = threadIdx.x * 4; j < d; j += 256 * 4) {
    const float4 v = *(const float4*)(row + j);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float rstd = 1.0f / sqrtf(tot / (float)d + eps);
  f16* o = out + (size_t)i * ldo;
  for (int j = threadIdx.x * 4; j < d; j += 256 * 4) {
    const float4 v = *(const float4*)(row + j);
    const float4 gm = *(const float4*)(gamma + j);
    f16x4 h = {(f16)(v.x * rstd * gm.x), (f16)(v.y * rstd * gm.y), (f16)(v.z * rstd * gm.z),
               (f16)(v.w * rstd * gm.w)};
    *(f16x4*)(o + j) = h;
  }
}

// The same with one wave per row and the row held in registers (NV float4
// per lane, d = 256 * NV), four rows per workgroup: every load of a row is in
// flight at once and the sum needs no LDS or barrier.  The sum of squares is
// reduced in a fixed order (lane order, then a butterfly over the wave).
template <int NV>
__global__ __launch_bounds__(256) void rmsnorm_wave_kernel(const float* __restrict__ x, int ldx,
                                                           const float* const* __restrict__ rowptr,
                                                           int R, const float* __restrict__ gamma,
                                                           float eps, f16* __restrict__ out,
                                                           int ldo) {
  constexpr int D = 256 * NV;
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= R) return;
  const float* row = rowptr ? rowptr[i] : x + (size_t)i * ldx;
  float4 v[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) v[j] = *(const float4*)(row + (j * 64 + lane) * 4);
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    ss += v[j].x * v[j].x;
    ss += v[j].y * v[j].y;
    ss += v[j].z * v[j].z;
    ss += v[j].w * v[j].w;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += shfl_xor(ss, o);
  const float rstd = 1.0f / sqrtf(ss / (float)D + eps);
  f16* o = out + (size_t)i * ldo;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int cix = (j * 64 + lane) * 4;
    const float4 gm = *(const float4*)(gamma + cix);
    *(f16x4*)(o + cix) = f16x4{(f16)(v[j].x * rstd * gm.x), (f16)(v[j].y * rstd * gm.y),
                              (f16)(v[j].z * rstd * gm.z), (f16)(v[j].w * rstd * gm.w)};
  }
}

// --------------------------------------------------------------- row gather
// Copies the residual row and the attention-output row of each selected token
// (the last token of every row, before the last layer's O-projection and MLP).
__global__ __launch_bounds__(256) void gather_rows_kernel(const int32_t* __restrict__ idx,
                                                          const float* __restrict__ x, int d,
                                                          float* __restrict__ x_out,
                                                          const f16* __restrict__ a, int da,
                                                          f16* __restrict__ a_out) {
  const int i = blockIdx.x;
  const size_t t = (size_t)idx[i];
  for (int j = threadIdx.x * 4; j < d; j += 256 * 4)
    *(float4*)(x_out + (size_t)i * d + j) = *(const float4*)(x + t * d + j);
  for (int j = threadIdx.x * 8; j < da; j += 256 * 8)
    *(f16x8*)(a_out + (size_t)i * da + j) = *(const f16x8*)(a + t * da + j);
}

// --------------------------------------------------------------- int4 repack
// One thread per (64-column block, group, lane, word): gathers the 8 codes of
// column nb*64 + 16f + c, features kg*32 + 8g .. +7, from its source row and
// writes them biased by +8 in the nibble order the GEMM's dequant expects.
__global__ void repack_kernel(RepackSrc src, const int32_t* __restrict__ colsrc, int np, int kg_n,
                              uint32_t* __restrict__ qpack, f16* __restrict__ spack) {
  const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)(np / 64) * kg_n * 256;
  if (item >= total) return;
  const int f = item & 3;
  const int lane = (item >> 2) & 63;
  const size_t blk = item >> 8;  // nb * kg_n + kg
  const int kg = (int)(blk % kg_n);
  const int nb = (int)(blk / kg_n);
  const int g = lane >> 4, c = lane & 15;
  const int col = nb * 64 + 16 * f + c;
  const int cs = colsrc[col];
  uint32_t word = 0x88888888u;  // code 0 everywhere
  f16 scale = (f16)0.0f;
  if (cs >= 0) {
    const int si = cs >> 24, r = cs & 0xFFFFFF;
    const int kp = src.kp_src[si];
    if (kg * 32 < kp) {
      const uint8_t* qb = src.q[si] + (size_t)r * (kp / 2) + kg * 16 + g * 4;
      uint32_t codes = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t nib = (qb[j >> 1] >> ((j & 1) * 4)) & 0xF;
        const uint32_t u = nib ^ 8u;  // two's complement -> biased
        const int p = (j & 1) ? 4 + (j >> 1) : (j >> 1);
        codes |= u << (4 * p);
      }
      word = codes;
      scale = ((const f16*)src.s[si])[(size_t)r * (kp / 32) + kg];
    }
  }
  qpack[item] = word;
  if (g == 0) spack[blk * 64 + c * 4 + f] = scale;
}

// One item per (64-column block, 32-feature group, half, lane): 16 bytes,
// the 8 codes of two columns.
__global__ void repack_fp8_kernel(RepackSrc src, const int32_t* __restrict__ colsrc, int np,
                                  int kg_n, uint8_t* __restrict__ qpack,
                                  float* __restrict__ sscale) {
  const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)(np / 64) * kg_n * 128;
  if (item >= total) return;
  const int lane = item & 63;
  const int h = (item >> 6) & 1;
  const size_t blk = item >> 7;  // nb * kg_n + kg
  const int kg = (int)(blk % kg_n);
  const int nb = (int)(blk / kg_n);
  const int g = lane >> 4, c = lane & 15;
  uint32_t w[4] = {0u, 0u, 0u, 0u};  // code 0 = +0.0
#pragma unroll
  for (int ff = 0; ff < 2; ++ff) {
    const int col = nb * 64 + 16 * (2 * h + ff) + c;
    const int cs = colsrc[col];
    float scale = 0.f;
    if (cs >= 0) {
      const int si = cs >> 24, r = cs & 0xFFFFFF;
      const int K = src.kp_src[si];
      const uint8_t* qr = src.q[si] + (size_t)r * K;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = kg * 32 + 8 * g + j;
        const uint32_t code = k < K ? qr[k] : 0u;
        w[2 * ff + (j >> 2)] |= code << (8 * (j & 3));
      }
      scale = src.sf[si][r];
    }
    if (kg == 0 && g == 0) sscale[col] = scale;
  }
  *(uint4*)(qpack + item * 16) = make_uint4(w[0], w[1], w[2], w[3]);
}

// --------------------------------------------------------------- head weight tiling
// One thread per 16-byte chunk of the tiled head weight: tile t, K step s,
// row r, chunk c holds features 32s + 8c .. +7 of vocabulary row 128t + r
// (zero past the vocabulary).
__global__ __launch_bounds__(256) void repack_head_kernel(const f16* __restrict__ src, int V,
                                                          int d, f16* __restrict__ dst,
                                                          size_t n_chunks) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_chunks) return;
  const int c = (int)(i & 3);
  const int r = (int)((i >> 2) % kHeadTileRows);
  const size_t ts = (i >> 2) / kHeadTileRows;  // tile * (d / 32) + step
  const int ks = (int)(ts % (size_t)(d / 32));
  const int v = (int)(ts / (size_t)(d / 32)) * kHeadTileRows + r;
  f16x8 x = {0, 0, 0, 0, 0, 0, 0, 0};
  if (v < V) x = *(const f16x8*)(src + (size_t)v * d + ks * 32 + c * 8);
  *(f16x8*)(dst + i * 8) = x;
}

// --------------------------------------------------------------- restricted head
// Logits of the allowed tokens only: one workgroup per row, one wave per
// allowed token at a time; each lane sums 8-feature runs with a stride of
// 512 features, then the wave adds the lanes in a fixed order.
__global__ __launch_bounds__(256) void head_restricted_kernel(const f16* __restrict__ hn, int d,
                                                              const f16* __restrict__ W,
                                                              const int32_t* __restrict__ allowed,
                                                              int n_sel, float* __restrict__ zsel,
                                                              float* __restrict__ dump,
                                                              int ld_dump) {
  const int r = blockIdx.x, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const f16* h = hn + (size_t)r * d;
  for (int i = wave; i < n_sel; i += 4) {
    const int tok = allowed[i];
    float acc = 0.f;
    for (int k = lane * 8; k < d; k += 512) {
      const f16x8 a = *(const f16x8*)(h + k);
      const f16x8 b = *(const f16x8*)(W + head_tiled_index(tok, k, d));
#pragma unroll
      for (int j = 0; j < 8; ++j) acc += (float)a[j] * (float)b[j];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc += shfl_xor(acc, o);
    if (lane == 0) {
      zsel[(size_t)r * n_sel + i] = acc;
      if (dump) dump[(size_t)r * ld_dump + tok] = acc;
    }
  }
}

// --------------------------------------------------------------- head finish
// One wave per row: LSE over the vocabulary from the per-slice partials, then
// the first maximum among the allowed tokens and the allowed-set LSE.  With a
// state mask the row's allowed tokens are the entries its state's mask row
// marks.
__global__ __launch_bounds__(64) void head_finalize_kernel(const float2* __restrict__ part,
                                                           int n_chunks,
                                                           const float* __restrict__ zsel,
                                                           int n_sel, int n_allowed,
                                                           const int32_t* __restrict__ allowed_tok,
                                                           HeadPick* __restrict__ out,
                                                           const int32_t* __restrict__ row_state,
                                                           const uint8_t* __restrict__ state_mask) {
  const int r = blockIdx.x, lane = threadIdx.x;
  const uint8_t* mk = state_mask ? state_mask + (size_t)row_state[r] * n_sel : nullptr;
  auto ok = [&](int j) { return mk == nullptr || mk[j] != 0; };
  const float2* pr = part + (size_t)r * n_chunks;
  float mx = -INFINITY;
  for (int j = lane; j < n_chunks; j += 64) mx = fmaxf(mx, pr[j].x);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, shfl_xor(mx, o));
  float sm = 0.f;
  for (int j = lane; j < n_chunks; j += 64) {
    const float2 v = pr[j];
    if (v.x > -INFINITY) sm += v.y * expf(v.x - mx);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) sm += shfl_xor(sm, o);
  const float lse_full = mx + logf(sm);

  const float* zr = zsel + (size_t)r * n_sel;
  // argmax with the smallest index on ties
  float best = -INFINITY;
  int bi = n_allowed;  // sentinel; stays only if every logit is NaN
  for (int j = lane; j < n_allowed; j += 64) {
    if (!ok(j)) continue;
    const float z = zr[j];
    if (z > best || (z == best && j < bi)) {
      best = z;
      bi = j;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ob = shfl_xor(best, o);
    const int oi = shfl_xor(bi, o);
    if (ob > best || (ob == best && oi < bi)) {
      best = ob;
      bi = oi;
    }
  }
  if (bi >= n_allowed) bi = 0;  // keeps the index in bounds whatever the logits hold
  float second = -INFINITY;
  int n_ok = 0;
  for (int j = lane; j < n_allowed; j += 64)
    if (ok(j)) {
      ++n_ok;
      if (j != bi) second = fmaxf(second, zr[j]);
    }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) second = fmaxf(second, shfl_xor(second, o));
  float sa = 0.f;
  for (int j = lane; j < n_allowed; j += 64)
    if (ok(j)) sa += expf(zr[j] - best);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    sa += shfl_xor(sa, o);
    n_ok += shfl_xor(n_ok, o);
  }
  if (lane == 0) {
    HeadPick hp;
    hp.index = bi;
    hp.token = allowed_tok[bi];
    hp.logprob = -logf(sa);
    hp.logprob_full = n_chunks > 0 ? best - lse_full : NAN;
    hp.margin = n_ok > 1 ? best - second : INFINITY;
    hp.pad[0] = hp.pad[1] = hp.pad[2] = 0.f;
    out[r] = hp;
  }
}

}  // namespace

hipError_t launch_fill_u32(hipStream_t s, void* p, size_t n_words, uint32_t value) {
  if (n_words == 0) return hipSuccess;
  if (((uintptr_t)p & 15) != 0) return hipErrorInvalidValue;
  const size_t groups = (n_words + 1023) / 1024;
  const int blocks = (int)(groups < 8192 ? groups : 8192);
  hipLaunchKernelGGL(fill_u32_kernel, dim3(blocks), dim3(256), 0, s, (uint32_t*)p, n_words, value);
  return hipGetLastError();
}

hipError_t launch_embed(hipStream_t s, const int32_t* tok, int T, const half_bits* emb, int d,
                        float* x) {
  if (T == 0) return hipSuccess;
  hipLaunchKernelGGL(embed_kernel, dim3(T), dim3(256), 0, s, tok, (const f16*)emb, d, x);
  return hipGetLastError();
}

hipError_t launch_gather_rows(hipStream_t s, const int32_t* idx, int R, const float* x, int d,
                              float* x_out, const half_bits* a, int da, half_bits* a_out) {
  if (R == 0) return hipSuccess;
  if (d % 4 != 0 || da % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(R), dim3(256), 0, s, idx, x, d, x_out,
                     (const f16*)a, da, (f16*)a_out);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(hipStream_t s, const float* x, int ldx, const float* const* rowptr,
                          int R, const float* gamma, int d, float eps, half_bits* out, int ldo) {
  if (R == 0) return hipSuccess;
  const dim3 g4((R + 3) / 4);
  switch (d) {  // the common model widths; others take the workgroup-per-row kernel
    case 256:
      hipLaunchKernelGGL(rmsnorm_wave_kernel<1>, g4, dim3(256), 0, s, x, ldx, rowptr, R, gamma, eps,
                         (f16*)out, ldo);
      break;
    case 2048:
      hipLaunchKernelGGL(rmsnorm_wave_kernel<8>, g4, dim3(256), 0, s, x, ldx, rowptr, R, gamma, eps,
                         (f16*)out, ldo);
      break;
    case 4096:
      hipLaunchKernelGGL(rmsnorm_wave_kernel<16>, g4, dim3(256), 0, s, x, ldx, rowptr, R, gamma,
                         eps, (f16*)out, ldo);
      break;
    default:
      hipLaunchKernelGGL(rmsnorm_kernel, dim3(R), dim3(256), 0, s, x, ldx, rowptr, gamma, d, eps,
                         (f16*)out, ldo);
  }
  return hipGetLastError();
}

hipError_t launch_repack_w4(hipStream_t s, const RepackSrc& src, const int32_t* colsrc,
                            PackedW& dst) {
  const int kg_n = dst.kp / 32;
  const size_t total = (size_t)(dst.np / 64) * kg_n * 256;
  const int blocks = (int)((total + 255) / 256);
  hipLaunchKernelGGL(repack_kernel, dim3(blocks), dim3(256), 0, s, src, colsrc, dst.np, kg_n,
                     dst.qpack, (f16*)dst.spack);
  return hipGetLastError();
}

hipError_t launch_repack_w8(hipStream_t s, const RepackSrc& src, const int32_t* colsrc,
                            PackedW& dst) {
  const int kg_n = dst.kp / 32;
  const size_t total = (size_t)(dst.np / 64) * kg_n * 128;
  const int blocks = (int)((total + 255) / 256);
  hipLaunchKernelGGL(repack_fp8_kernel, dim3(blocks), dim3(256), 0, s, src, colsrc, dst.np, kg_n,
                     (uint8_t*)dst.qpack, dst.sscale);
  return hipGetLastError();
}

hipError_t launch_repack_head(hipStream_t s, const half_bits* src, int V, int d, half_bits* dst) {
  if (d % 32 != 0) return hipErrorInvalidValue;
  const size_t vp = (size_t)(V + kHeadTileRows - 1) / kHeadTileRows * kHeadTileRows;
  const size_t n_chunks = vp * d / 8;
  const size_t blocks = (n_chunks + 255) / 256;
  hipLaunchKernelGGL(repack_head_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     (const f16*)src, V, d, (f16*)dst, n_chunks);
  return hipGetLastError();
}

hipError_t launch_head_restricted(hipStream_t s, const half_bits* hn, int R, int d,
                                  const half_bits* W, const int32_t* allowed, int n_sel,
                                  float* zsel, float* dump, int ld_dump) {
  if (R == 0 || n_sel == 0) return hipSuccess;
  if (d % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(head_restricted_kernel, dim3(R), dim3(256), 0, s, (const f16*)hn, d,
                     (const f16*)W, allowed, n_sel, zsel, dump, ld_dump);
  return hipGetLastError();
}

hipError_t launch_head_finalize(hipStream_t s, const float2* part, int n_chunks,
                                const float* zsel, int n_sel, int n_allowed,
                                const int32_t* allowed_tok, int R, HeadPick* out,
                                const int32_t* row_state, const uint8_t* state_mask) {
  if (R == 0) return hipSuccess;
  if (state_mask && !row_state) return hipErrorInvalidValue;
  hipLaunchKernelGGL(head_finalize_kernel, dim3(R), dim3(64), 0, s, part, n_chunks, zsel, n_sel,
                     n_allowed, allowed_tok, out, row_state, state_mask);
  return hipGetLastError();
}

}  // namespace lmop
