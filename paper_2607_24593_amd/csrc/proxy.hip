// Proxy aggregation (Sec. 4.2 Eq. 4): the per-head mean of a group's
// dequantised queries and of its gates, stored back in the query format.
//
// One workgroup per group, 256 threads x 32 consecutive elements of the
// 64 x 128 row.  Every step is rounded once in fp32, in a fixed order
// (member-ascending sums, then one correctly rounded divide by |G|), with FMA
// contraction disabled, so the result is reproducible bit for bit:
//   fp8 : mean of (qscale_t * q8_t); scale = amax / 448; codes = RNE(mean / scale)
//   bf16: mean of q_t; RNE to bf16
// A group of one is copied unchanged, and so is the chosen member for the
// first / last aggregation (Sec. 5.4).  For fp8 the kernel can also write the
// score epilogue's linear terms (lin_row) of the proxy and of the members,
// which saves a pass over the member rows.
#include <algorithm>

#include "dpp.h"
#include "launch.h"
#include "mfma_tile.h"
#include "pivot.h"

namespace pivot {

// Four fp32 -> E4M3FN codes packed little-endian, round to nearest even
// (gfx950 OCP conversion).
__device__ __forceinline__ uint32_t encode_e4m3_quad(float a, float b, float c, float d) {
  int word = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c, d, word, true);
}

__device__ __forceinline__ float decode_e4m3(uint32_t word, int byte) {
  // byte is a compile-time constant after unrolling
  switch (byte) {
    case 0: return __builtin_amdgcn_cvt_f32_fp8((int)word, 0);
    case 1: return __builtin_amdgcn_cvt_f32_fp8((int)word, 1);
    case 2: return __builtin_amdgcn_cvt_f32_fp8((int)word, 2);
    default: return __builtin_amdgcn_cvt_f32_fp8((int)word, 3);
  }
}

// a / b rounded once, from y = RN(1 / b) (Markstein's division step): q0 =
// RN(a y) lies within an ulp of a / b, so the remainder q0 b - a is exact and
// q0 - (q0 b - a) y rounds to RN(a / b).  Taking the remainder as q0 b - a
// keeps the sign of a zero quotient.  For b in [2^-80, 2^100] this is a / b
// rounded once whenever |a / b| >= 2^-11 (a is then at least 2^-91, far from
// the subnormals where the remainder could round); a smaller quotient may be
// an ulp off, and both round to the same signed zero in E4M3.  Three VALU
// operations in place of the eleven of a general fp32 divide.
__device__ __forceinline__ float div_rn(float a, float b, float y) {
  const float q0 = a * y;
  return fmaf(fmaf(q0, b, -a), -y, q0);
}
__device__ __forceinline__ bool div_rn_ok(float b) { return b >= 0x1p-80f && b <= 0x1p100f; }

// The linear part of the fp8 epilogue (mfma_tile.h) for one row, by one wave:
// u = sum_j (w_j * qscale / 2) * q8_j, a 128-vector, stored as four fp8
// levels: level l holds codes c_l = RNE((u - sum_{l'<l} sigma_l' c_l') /
// sigma_l) with sigma_0 = max|u| / 448 and sigma_l = sigma_0 16^-l.  No level
// saturates (a residual is at most half a code step of the level before,
// <= 256 sigma_l), and the last residual is at most sigma_0 / 1024, about
// 2^-19 of max|u|.  The fixed ratio leaves one scale per row for the
// epilogue; out_scale still receives all four.
// Lane l reads the 16-byte slices (dims 16 (l / 8) ..) of heads l % 8,
// l % 8 + 8, ..: eight loads per lane, all in flight at once.  The eight
// partial sums of a dim are then added across lanes (xor 1, 2, 4, as DPP
// steps) in a fixed order, halving the vector at each step, so that lane l
// ends with dims 2l and 2l+1 to quantise.  qr and wr may point to global
// memory or LDS.  Every operation is explicit (no contraction), so each
// caller gets the same bits.
__device__ __forceinline__ void lin_row(const uint8_t* qr, const float* wr, float qscale, uint8_t* out,
                                        float* out_scale, int lane) {
#pragma clang fp contract(off)
  const float half_scale = qscale * 0.5f;
  const int hs = lane & 7, db = lane >> 3;
  uint4 v[8];
  float wh[8];
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int h = 8 * it + hs;
    v[it] = *reinterpret_cast<const uint4*>(qr + h * kD + 16 * db);
    wh[it] = wr[h];
  }
  float u[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) u[e] = 0.f;
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const float x = wh[it] * half_scale;
    const uint32_t words[4] = {v[it].x, v[it].y, v[it].z, v[it].w};
#pragma unroll
    for (int e = 0; e < 16; ++e) u[e] = fmaf(x, decode_e4m3(words[e >> 2], e & 3), u[e]);
  }
  // Reduce-scatter over the 8 lanes hs of a dim block.  After the xor-1 step
  // a lane keeps the elements whose bit 1 equals its hs bit 0, after xor 2
  // those whose bit 2 equals hs bit 1, after xor 4 bit 3 = hs bit 2: lane hs
  // is left with elements 2 hs and 2 hs + 1.  Every add takes the same two
  // partial sums as a full butterfly, so the bits are unchanged.
  const bool h0 = hs & 1, h1 = hs & 2, h2 = hs & 4;
  float s8[8];  // index (e3 e2 e0)
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int lo = ((i & 6) << 1) | (i & 1);  // element with bit 1 clear
    const float keep = h0 ? u[lo | 2] : u[lo], send = h0 ? u[lo] : u[lo | 2];
    s8[i] = keep + lane_xor1(send);
  }
  float s4[4];  // index (e3 e0)
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int lo = ((j & 2) << 1) | (j & 1);  // s8 index with e2 clear
    const float keep = h1 ? s8[lo | 2] : s8[lo], send = h1 ? s8[lo] : s8[lo | 2];
    s4[j] = keep + lane_xor2(send);
  }
  float u0, u1;
  {
    const float keep0 = h2 ? s4[2] : s4[0], send0 = h2 ? s4[0] : s4[2];
    const float keep1 = h2 ? s4[3] : s4[1], send1 = h2 ? s4[1] : s4[3];
    u0 = keep0 + lane_xor4(send0);
    u1 = keep1 + lane_xor4(send1);
  }
  const float amax = wave_reduce(fmaxf(fabsf(u0), fabsf(u1)), [](float a, float b) { return fmaxf(a, b); });
  const float sigma0 = amax > 0.f ? amax / 448.0f : 1.0f;
  const float y0 = 1.0f / sigma0;
  auto level = [&](int l, float q0, float q1) {
    const float sigma = sigma0 * kLinStep[l];  // exact: a power of two
    const int word = __builtin_amdgcn_cvt_pk_fp8_f32(q0, q1, 0, false);
    *reinterpret_cast<uint16_t*>(out + l * kD + 2 * lane) = (uint16_t)word;
    u0 = u0 - sigma * __builtin_amdgcn_cvt_f32_fp8(word, 0);
    u1 = u1 - sigma * __builtin_amdgcn_cvt_f32_fp8(word, 1);
    if (lane == 0) out_scale[l] = sigma;
  };
  if (div_rn_ok(sigma0) && div_rn_ok(sigma0 * kLinStep[kLinLevels - 1])) {
#pragma unroll
    for (int l = 0; l < kLinLevels; ++l) {
      const float sigma = sigma0 * kLinStep[l], y = y0 * (float)(1 << (4 * l));  // both exact
      level(l, div_rn(u0, sigma, y), div_rn(u1, sigma, y));
    }
  } else {
#pragma unroll
    for (int l = 0; l < kLinLevels; ++l) {
      const float sigma = sigma0 * kLinStep[l];
      level(l, u0 / sigma, u1 / sigma);
    }
  }
}

template <int DT>
__global__ __launch_bounds__(256) void proxy_kernel(const uint8_t* __restrict__ q,
                                                    const float* __restrict__ q_scale,
                                                    const float* __restrict__ w, int g, SeqTable st, int j0,
                                                    int all_groups, int agg,
                                                    uint8_t* __restrict__ pq, float* __restrict__ psc,
                                                    float* __restrict__ pw, LinOut lo, int stage) {
#pragma clang fp contract(off)
  // stage (fp8, members' linear terms wanted, g <= MB): the mean pass copies
  // each member row it loads into dynamic LDS (g x 8 KiB), and the members'
  // linear terms are computed from there rather than read again from HBM;
  // their gates follow the rows (g x 256 B).  The proxy's codes, for its own linear term, take the region's first 8 KiB
  // (member 0's slot, once the members' terms are done), so a workgroup of
  // four members holds 33 KiB and four fit a CU.
  extern __shared__ uint4 mrows[];
  constexpr int EB = DT == kFp8 ? 1 : 2;
  constexpr int ROW_BYTES = kH * kD * EB;
  float* const mgates = reinterpret_cast<float*>(mrows + g * (ROW_BYTES / 16));
  constexpr int PER = 32;  // elements per thread
  const int j = j0 + blockIdx.x, b = blockIdx.y;
  if (b >= st.n || j >= seq_groups(st, b, g)) return;
  if (!all_groups && j < st.first_proxy[b]) return;
  const int gs = min(g, st.n_rows[b] - j * g);
  const int64_t r0 = (int64_t)st.row0[b] + (int64_t)j * g;
  const int64_t pr = (int64_t)st.grp0[b] + j;
  const int tid = threadIdx.x;
  const int e0 = tid * PER;

  if (gs == 1 || agg != PIVOT_AGG_MEAN) {
    const int64_t rc = r0 + (agg == PIVOT_AGG_LAST ? gs - 1 : 0);
    const uint4* src = reinterpret_cast<const uint4*>(q + rc * ROW_BYTES + e0 * EB);
    uint4* dst = reinterpret_cast<uint4*>(pq + pr * ROW_BYTES + e0 * EB);
#pragma unroll
    for (int v = 0; v < PER * EB / 16; ++v) dst[v] = src[v];
    if (tid == 0) psc[pr] = (DT == kFp8) ? q_scale[rc] : 1.0f;
    if (tid < kH) pw[pr * kH + tid] = w[rc * kH + tid];
    if constexpr (DT == kFp8) {
      const int wave = tid >> 6, lane = tid & 63;
      if (lo.plin && wave == (gs & 3))  // the proxy's linear term: that of row rc
        lin_row(q + rc * ROW_BYTES, w + rc * kH, q_scale[rc], lo.plin + pr * kLinBytes, lo.plsc + pr * kLinLevels,
                lane);
      if (lo.qlin)
        for (int r = wave; r < gs; r += 4)
          lin_row(q + (r0 + r) * ROW_BYTES, w + (r0 + r) * kH, q_scale[r0 + r], lo.qlin + (r0 + r) * kLinBytes,
                  lo.qlsc + (r0 + r) * kLinLevels, lane);
    }
    return;
  }

  // Members are read MB at a time: every load of a batch is issued before the
  // first is used, then the batch is summed in ascending member order.
  constexpr int VPM = PER * EB / 16;      // 16-byte loads per member and thread
  constexpr int MB = DT == kFp8 ? 8 : 4;  // members per batch
  float sum[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) sum[e] = 0.0f;
  float wsum = 0.0f;
  for (int u0 = 0; u0 < gs; u0 += MB) {
    uint4 v[MB][VPM];
    float sq[MB], wv[MB];
#pragma unroll
    for (int k = 0; k < MB; ++k) {
      const int64_t row = r0 + u0 + k;
      if (u0 + k < gs) {
        const uint4* src = reinterpret_cast<const uint4*>(q + row * ROW_BYTES + e0 * EB);
#pragma unroll
        for (int x = 0; x < VPM; ++x) v[k][x] = src[x];
        sq[k] = (DT == kFp8) ? q_scale[row] : 1.0f;
        wv[k] = tid < kH ? w[row * kH + tid] : 0.0f;
      }
    }
    if (stage) {  // one batch holds every member (g <= MB)
#pragma unroll
      for (int k = 0; k < MB; ++k)
        if (k < gs)
#pragma unroll
          for (int x = 0; x < VPM; ++x) mrows[k * (ROW_BYTES / 16) + VPM * tid + x] = v[k][x];
      if (tid < kH)
#pragma unroll
        for (int k = 0; k < MB; ++k)
          if (k < gs) mgates[k * kH + tid] = wv[k];
    }
#pragma unroll
    for (int k = 0; k < MB; ++k) {
      if (u0 + k >= gs) break;
      wsum = wsum + wv[k];
      if constexpr (DT == kFp8) {
        const uint32_t words[8] = {v[k][0].x, v[k][0].y, v[k][0].z, v[k][0].w,
                                   v[k][1].x, v[k][1].y, v[k][1].z, v[k][1].w};
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          float x = decode_e4m3(words[e >> 2], e & 3);
          float deq = sq[k] * x;
          sum[e] = sum[e] + deq;
        }
      } else {
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const uint32_t words[4] = {v[k][x].x, v[k][x].y, v[k][x].z, v[k][x].w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            sum[8 * x + 2 * h] = sum[8 * x + 2 * h] + __uint_as_float(words[h] << 16);
            sum[8 * x + 2 * h + 1] = sum[8 * x + 2 * h + 1] + __uint_as_float(words[h] & 0xFFFF0000u);
          }
        }
      }
    }
  }
  const float count = (float)gs;
  // correctly rounded fp32 divides; by a power of two the product with its
  // exact reciprocal is the same correctly rounded value
  if ((gs & (gs - 1)) == 0) {
    const float inv = 1.0f / count;
#pragma unroll
    for (int e = 0; e < PER; ++e) sum[e] = sum[e] * inv;
    wsum = wsum * inv;
  } else {
#pragma unroll
    for (int e = 0; e < PER; ++e) sum[e] = sum[e] / count;
    wsum = wsum / count;
  }
  float amax = 0.0f;
#pragma unroll
  for (int e = 0; e < PER; ++e) amax = fmaxf(amax, fabsf(sum[e]));

  if (tid < kH) pw[pr * kH + tid] = wsum;

  if constexpr (DT == kFp8) {
    __shared__ float wmax[4];
    amax = wave_reduce(amax, [](float a, float b) { return fmaxf(a, b); });
    if ((tid & 63) == 0) wmax[tid >> 6] = amax;
    __syncthreads();
    amax = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
    const float sigma = amax > 0.0f ? amax / 448.0f : 1.0f;
    uint32_t out[8];
    if (div_rn_ok(sigma)) {  // uniform over the workgroup
      const float y = 1.0f / sigma;
#pragma unroll
      for (int v = 0; v < 8; ++v)
        out[v] = encode_e4m3_quad(div_rn(sum[4 * v], sigma, y), div_rn(sum[4 * v + 1], sigma, y),
                                  div_rn(sum[4 * v + 2], sigma, y), div_rn(sum[4 * v + 3], sigma, y));
    } else {
#pragma unroll
      for (int v = 0; v < 8; ++v)
        out[v] = encode_e4m3_quad(sum[4 * v] / sigma, sum[4 * v + 1] / sigma, sum[4 * v + 2] / sigma,
                                  sum[4 * v + 3] / sigma);
    }
    uint4* dst = reinterpret_cast<uint4*>(pq + pr * ROW_BYTES + e0);
    dst[0] = uint4{out[0], out[1], out[2], out[3]};
    dst[1] = uint4{out[4], out[5], out[6], out[7]};
    if (tid == 0) psc[pr] = sigma;
    // the linear terms: the members' (Refine re-scores them) from their rows,
    // which this workgroup has just read, then the proxy's from its codes and
    // gates staged in LDS
    const int wave = tid >> 6, lane = tid & 63;
    if (lo.qlin)  // the staged rows were written before the amax barrier above
      for (int r = wave; r < gs; r += 4)
        lin_row(stage ? reinterpret_cast<const uint8_t*>(mrows + r * (ROW_BYTES / 16)) : q + (r0 + r) * ROW_BYTES,
                stage ? mgates + r * kH : w + (r0 + r) * kH, q_scale[r0 + r], lo.qlin + (r0 + r) * kLinBytes, lo.qlsc + (r0 + r) * kLinLevels,
                lane);
    if (lo.plin) {
      uint4* prow = mrows;  // member 0's staged row is no longer read past the barrier
      __shared__ float pws[kH];
      if (stage) __syncthreads();
      prow[2 * tid] = uint4{out[0], out[1], out[2], out[3]};
      prow[2 * tid + 1] = uint4{out[4], out[5], out[6], out[7]};
      if (tid < kH) pws[tid] = wsum;
      __syncthreads();
      if (wave == (gs & 3))
        lin_row(reinterpret_cast<const uint8_t*>(prow), pws, sigma, lo.plin + pr * kLinBytes,
                lo.plsc + pr * kLinLevels, lane);
    }
  } else {
    uint32_t out[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) out[v] = (uint32_t)bf16_rne(sum[2 * v]) | ((uint32_t)bf16_rne(sum[2 * v + 1]) << 16);
    uint4* dst = reinterpret_cast<uint4*>(pq + pr * ROW_BYTES + e0 * 2);
#pragma unroll
    for (int v = 0; v < 4; ++v) dst[v] = uint4{out[4 * v], out[4 * v + 1], out[4 * v + 2], out[4 * v + 3]};
    if (tid == 0) psc[pr] = 1.0f;
  }
}

hipError_t launch_proxy(int dtype, const void* q, const float* q_scale, const float* w, int g, const SeqTable& st,
                        int j0, int j1, bool all_groups, int agg, void* pq, float* psc, float* pw, hipStream_t stream,
                        const LinOut& lo) {
  if (dtype != kFp8 && (lo.plin || lo.qlin)) return hipErrorInvalidValue;  // linear terms are fp8 only
  if (j1 <= j0 || st.n <= 0) return hipSuccess;
  dim3 grid((unsigned)(j1 - j0), (unsigned)st.n);
  // members staged in LDS for their linear terms when one load batch holds a group
  const int stage = dtype == kFp8 && lo.qlin && agg == PIVOT_AGG_MEAN && g > 1 && g <= 8;
  // dynamic LDS: the staged members and their gates, and the proxy's codes (in the first slot)
  const size_t shmem =
      std::max(stage ? (size_t)g * (kH * kD + kH * sizeof(float)) : 0, dtype == kFp8 && lo.plin ? (size_t)kH * kD : 0);
  if (dtype == kFp8)
    hipLaunchKernelGGL(proxy_kernel<kFp8>, grid, dim3(256), shmem, stream, (const uint8_t*)q, q_scale, w, g, st, j0,
                       (int)all_groups, agg, (uint8_t*)pq, psc, pw, lo, stage);
  else
    hipLaunchKernelGGL(proxy_kernel<kBf16>, grid, dim3(256), 0, stream, (const uint8_t*)q, q_scale, w, g, st, j0,
                       (int)all_groups, agg, (uint8_t*)pq, psc, pw, LinOut{}, 0);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void encode_e4m3_kernel(const float* __restrict__ x, uint8_t* __restrict__ out,
                                                          int64_t n) {
  int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = (i + e < n) ? x[i + e] : 0.0f;
  uint32_t word = encode_e4m3_quad(v[0], v[1], v[2], v[3]);
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (i + e < n) out[i + e] = (uint8_t)(word >> (8 * e));
}

hipError_t launch_encode_e4m3(const float* x, uint8_t* out, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 1023) / 1024;
  hipLaunchKernelGGL(encode_e4m3_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, x, out, n);
  return hipGetLastError();
}

}  // namespace pivot

namespace pivot {

// Linear terms (lin_row) of flat row ranges, one wave per row.
__global__ __launch_bounds__(256) void lin_kernel(LinRows set0, LinRows set1, int64_t blocks0) {
  const bool first = blockIdx.x < blocks0;
  const LinRows rs = first ? set0 : set1;
  const int64_t row = rs.r0 + ((int64_t)blockIdx.x - (first ? 0 : blocks0)) * 4 + (threadIdx.x >> 6);
  if (row >= rs.r1) return;
  lin_row(rs.q + row * (int64_t)(kH * kD), rs.w + row * kH, rs.q_scale[row], rs.lin + row * (int64_t)kLinBytes,
          rs.lin_scale + row * kLinLevels, threadIdx.x & 63);
}

hipError_t launch_lin(const LinRows& set0, const LinRows& set1, hipStream_t stream) {
  const int64_t b0 = set0.r1 > set0.r0 ? (set0.r1 - set0.r0 + 3) / 4 : 0;
  const int64_t b1 = set1.r1 > set1.r0 ? (set1.r1 - set1.r0 + 3) / 4 : 0;
  if (b0 + b1 == 0) return hipSuccess;
  if (b0 + b1 > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(lin_kernel, dim3((unsigned)(b0 + b1)), dim3(256), 0, stream, set0, set1, b0);
  return hipGetLastError();
}

hipError_t launch_lin(const void* q, const float* q_scale, const float* w, int64_t r0, int64_t r1, uint8_t* lin,
                      float* lin_scale, hipStream_t stream) {
  return launch_lin(LinRows{(const uint8_t*)q, q_scale, w, r0, r1, lin, lin_scale}, LinRows{}, stream);
}

}  // namespace pivot
