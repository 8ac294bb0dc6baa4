// Producer of the computed tokens' Q/K/V: projection of their hidden states and rotary
// position embedding (the attention inputs of a prefill; the paper serves Qwen3-14B, Sec. 4,
// and the layer details follow its public configuration).
//
//   y = x W^T            x [T][H] bf16, W [(Hq + 2 Hkv) D][H] bf16, y bf16 (fp32 accumulate)
//   q, k = rotary(y_q, y_k) at each token's absolute position; v = y_v
//
// The projection is a plain GEMM and goes to rocBLAS (bf16 in/out, fp32 compute).  One
// work-group per token then reads the token's y row once: it finds the token's position from
// cu_q / seq_lens (suffix token i of request r sits at L_r - S_r + i), computes the D/2 rotary
// angles p * theta^(-2i/D) in fp64, reduced mod 2 pi before the fp32 sine and cosine, rotates
// the (i, i + D/2) pairs of every query and key head in fp32 and writes bf16 (round to
// nearest even) Q [T][Hq][D], K [T][Hkv][D] and V [T][Hkv][D]; K and V then go to the pool
// through the KV scatter.
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <cmath>
#include <mutex>

#include "../host/internal.hpp"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {  // nearest even; inputs finite
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

template <int D>
__global__ __launch_bounds__(kThreads) void qkv_rope_kernel(
    const uint16_t* __restrict__ y, int hq, int hkv, const int32_t* __restrict__ cu_q,
    const int32_t* __restrict__ seq_lens, int n_reqs, double theta, uint16_t* __restrict__ q_out,
    uint16_t* __restrict__ k_out, uint16_t* __restrict__ v_out) {
  constexpr int HALF = D / 2;
  __shared__ float cs[HALF], sn[HALF];
  __shared__ int pos_s;
  const int64_t t = blockIdx.x;
  const int tid = threadIdx.x;
  if (tid == 0) {  // request of token t: the last r with cu_q[r] <= t
    int lo = 0, hi = n_reqs - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) / 2;
      if (cu_q[mid] <= t) lo = mid; else hi = mid - 1;
    }
    pos_s = seq_lens[lo] - (cu_q[lo + 1] - cu_q[lo]) + static_cast<int>(t - cu_q[lo]);
  }
  __syncthreads();
  const double p = static_cast<double>(pos_s);
  for (int i = tid; i < HALF; i += kThreads) {
    const double a = std::fmod(p * std::pow(theta, -2.0 * i / D), 6.283185307179586476925);
    float s, c;
    sincosf(static_cast<float>(a), &s, &c);
    cs[i] = c;
    sn[i] = s;
  }
  __syncthreads();
  const int nrot = hq + hkv;
  const uint16_t* row = y + t * static_cast<int64_t>(hq + 2 * hkv) * D;
  for (int e = tid; e < nrot * HALF; e += kThreads) {
    const int h = e / HALF, i = e % HALF;
    const float lo = bf16_to_f32(row[h * D + i]), hi = bf16_to_f32(row[h * D + i + HALF]);
    uint16_t* dst = h < hq ? q_out + (t * hq + h) * D : k_out + (t * hkv + (h - hq)) * D;
    dst[i] = f32_to_bf16(lo * cs[i] - hi * sn[i]);
    dst[i + HALF] = f32_to_bf16(hi * cs[i] + lo * sn[i]);
  }
  const uint16_t* vrow = row + static_cast<int64_t>(nrot) * D;
  for (int e = tid; e < hkv * D; e += kThreads) v_out[t * hkv * D + e] = vrow[e];
}

// One rocBLAS handle per device, created on first use and kept for the process.
rocblas_handle blas_handle(int32_t* status) {
  static std::mutex mu;
  static rocblas_handle handles[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    *status = arckv::fail(ARCKV_EDEVICE, "qkv_rope: no current device");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (handles[dev] == nullptr && rocblas_create_handle(&handles[dev]) != rocblas_status_success) {
    handles[dev] = nullptr;
    *status = arckv::fail(ARCKV_EDEVICE, "qkv_rope: rocblas_create_handle failed");
    return nullptr;
  }
  *status = ARCKV_OK;
  return handles[dev];
}

}  // namespace

extern "C" int32_t arckv_qkv_rope(const void* x, const void* w_qkv, int64_t n_tokens, int32_t hidden,
                                  int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                  const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs,
                                  double rope_theta, void* y_workspace, int64_t ws_bytes, void* q_out,
                                  void* k_out, void* v_out, void* stream) {
  if (n_tokens < 0 || hidden < 1 || num_q_heads < 1 || num_kv_heads < 1 || n_reqs < 0 ||
      num_q_heads % num_kv_heads != 0 || !(rope_theta > 1.0) || !std::isfinite(rope_theta))
    return arckv::fail(ARCKV_EINVAL, "qkv_rope: bad sizes or theta");
  if (head_dim != 64 && head_dim != 128)
    return arckv::fail(ARCKV_EUNSUPPORTED, "qkv_rope: head_dim %d not in {64,128}", head_dim);
  if (n_tokens == 0) return ARCKV_OK;
  const int64_t n_out = static_cast<int64_t>(num_q_heads + 2 * num_kv_heads) * head_dim;
  if (n_tokens > INT32_MAX || n_out > INT32_MAX || n_reqs < 1)
    return arckv::fail(ARCKV_EINVAL, "qkv_rope: %lld tokens, %lld outputs, %d requests",
                       (long long)n_tokens, (long long)n_out, n_reqs);
  if (x == nullptr || w_qkv == nullptr || cu_q == nullptr || seq_lens == nullptr ||
      y_workspace == nullptr || q_out == nullptr || k_out == nullptr || v_out == nullptr)
    return arckv::fail(ARCKV_EINVAL, "qkv_rope: NULL pointer");
  if (ws_bytes < n_tokens * n_out * 2)
    return arckv::fail(ARCKV_ENOSPC, "qkv_rope: workspace %lld bytes < %lld", (long long)ws_bytes,
                       (long long)(n_tokens * n_out * 2));
  int32_t st = ARCKV_OK;
  rocblas_handle h = blas_handle(&st);
  if (h == nullptr) return st;
  auto* s = static_cast<hipStream_t>(stream);
  if (rocblas_set_stream(h, s) != rocblas_status_success)
    return arckv::fail(ARCKV_EDEVICE, "qkv_rope: rocblas_set_stream failed");
  // row-major y [T][N] = x [T][H] . W^T, W [N][H]: column-major y^T (N x T) = W^T-view op
  const float alpha = 1.0f, beta = 0.0f;
  const rocblas_status bs = rocblas_gemm_ex(
      h, rocblas_operation_transpose, rocblas_operation_none, static_cast<rocblas_int>(n_out),
      static_cast<rocblas_int>(n_tokens), hidden, &alpha, w_qkv, rocblas_datatype_bf16_r, hidden, x,
      rocblas_datatype_bf16_r, hidden, &beta, y_workspace, rocblas_datatype_bf16_r,
      static_cast<rocblas_int>(n_out), y_workspace, rocblas_datatype_bf16_r,
      static_cast<rocblas_int>(n_out), rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  if (bs != rocblas_status_success)
    return arckv::fail(ARCKV_EDEVICE, "qkv_rope: rocblas_gemm_ex status %d", static_cast<int>(bs));
  const dim3 grid(static_cast<unsigned>(n_tokens));
  auto* y = static_cast<const uint16_t*>(y_workspace);
  auto* q = static_cast<uint16_t*>(q_out);
  auto* k = static_cast<uint16_t*>(k_out);
  auto* v = static_cast<uint16_t*>(v_out);
  if (head_dim == 64)
    hipLaunchKernelGGL(qkv_rope_kernel<64>, grid, dim3(kThreads), 0, s, y, num_q_heads, num_kv_heads,
                       cu_q, seq_lens, n_reqs, rope_theta, q, k, v);
  else
    hipLaunchKernelGGL(qkv_rope_kernel<128>, grid, dim3(kThreads), 0, s, y, num_q_heads, num_kv_heads,
                       cu_q, seq_lens, n_reqs, rope_theta, q, k, v);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return arckv::fail(ARCKV_EDEVICE, "qkv_rope: %s", hipGetErrorString(e));
  return ARCKV_OK;
}
