// Elementwise steps of the full counter-causal pass (Sec. 3.1: every layer runs with fresh
// queries at the original position ids against the stored keys/values): the embedding
// gather into the fp32 residual stream, RMSNorm to the bf16 GEMM input, and the rotary
// angle table.  The GEMMs (with RoPE / residual / SwiGLU epilogues) live in gemm.hip.
#include "cc_internal.h"

namespace cc {
namespace {

constexpr int RNT = 256;

__global__ __launch_bounds__(RNT) void embed_kernel(const u16* __restrict__ embed,
                                                    const int32_t* __restrict__ ids,
                                                    float* __restrict__ h, int D) {
  const int n = blockIdx.x;
  const u16* row = embed + int64_t(ids ? ids[n] : n) * D;   // no ids: widen row n
  float* out = h + int64_t(n) * D;
  for (int i = threadIdx.x * 4; i < D; i += RNT * 4) {
    const uint2 v = *reinterpret_cast<const uint2*>(row + i);
    float4 f;
    f.x = __uint_as_float(v.x << 16);
    f.y = __uint_as_float(v.x & 0xffff0000u);
    f.z = __uint_as_float(v.y << 16);
    f.w = __uint_as_float(v.y & 0xffff0000u);
    *reinterpret_cast<float4*>(out + i) = f;
  }
}

// One workgroup per entry; D is a multiple of 4.
__global__ __launch_bounds__(RNT) void rmsnorm_kernel(const float* __restrict__ h,
                                                      const u16* __restrict__ gamma,
                                                      u16* __restrict__ y, int D, float eps) {
  __shared__ float wsum[RNT / 64];
  const int n = blockIdx.x;
  const float* x = h + int64_t(n) * D;
  float ss = 0.f;
  for (int i = threadIdx.x * 4; i < D; i += RNT * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + i);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < RNT / 64; ++w) tot += wsum[w];
  const float r = rsqrtf(tot / float(D) + eps);
  u16* out = y + int64_t(n) * D;
  for (int i = threadIdx.x * 4; i < D; i += RNT * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + i);
    const uint2 gm = *reinterpret_cast<const uint2*>(gamma + i);
    const float g0 = __uint_as_float(gm.x << 16), g1 = __uint_as_float(gm.x & 0xffff0000u);
    const float g2 = __uint_as_float(gm.y << 16), g3 = __uint_as_float(gm.y & 0xffff0000u);
    uint2 o;
    o.x = pack_bf2(v.x * r * g0, v.y * r * g1);
    o.y = pack_bf2(v.z * r * g2, v.w * r * g3);
    *reinterpret_cast<uint2*>(out + i) = o;
  }
}

// One thread per (entry, frequency).  The angle is formed and reduced in fp64 so large
// positions keep full fp32 accuracy in cos/sin.
__global__ void rope_table_kernel(const int32_t* __restrict__ pos, const int32_t* __restrict__ cu,
                                  int n_seqs, float2* __restrict__ rot, int N, int half,
                                  double theta, int head_dim) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= int64_t(N) * half) return;
  const int n = int(idx / half), e = int(idx % half);
  int p;
  if (pos) {
    p = pos[n];
  } else {
    int lo = 0, hi = n_seqs - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cu[mid] <= n) lo = mid; else hi = mid - 1;
    }
    p = n - cu[lo];
  }
  const double inv = pow(theta, -2.0 * double(e) / double(head_dim));
  double sn, cs;
  sincos(double(p) * inv, &sn, &cs);
  rot[idx] = make_float2(float(cs), float(sn));
}

}  // namespace

hipError_t launch_embed(const void* embed, const int32_t* ids, float* h, int N, int D,
                        hipStream_t s) {
  if (N == 0) return hipSuccess;
  hipLaunchKernelGGL(embed_kernel, dim3(N), dim3(RNT), 0, s, static_cast<const u16*>(embed), ids,
                     h, D);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const float* h, const void* gamma, void* y, int N, int D, float eps,
                          hipStream_t s) {
  if (N == 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(N), dim3(RNT), 0, s, h, static_cast<const u16*>(gamma),
                     static_cast<u16*>(y), D, eps);
  return hipGetLastError();
}

hipError_t launch_rope_table(const int32_t* pos, const int32_t* cu, int n_seqs, float2* rot, int N,
                             int head_dim, double theta, hipStream_t s) {
  if (N == 0) return hipSuccess;
  const int half = head_dim / 2;
  const int64_t total = int64_t(N) * half;
  hipLaunchKernelGGL(rope_table_kernel, dim3(unsigned((total + 255) / 256)), dim3(256), 0, s, pos,
                     cu, n_seqs, rot, N, half, theta, head_dim);
  return hipGetLastError();
}

}  // namespace cc
