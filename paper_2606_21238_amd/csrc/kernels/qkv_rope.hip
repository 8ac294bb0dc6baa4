// Producer of the computed tokens' Q/K/V: projection of their hidden states and rotary
// position embedding (the attention inputs of a prefill; the paper serves Qwen3-14B, Sec. 4,
// and the layer details follow its public configuration).
//
//   y = x W^T            x [T][H] bf16, W [(Hq + 2 Hkv) D][H] bf16, y bf16 (fp32 accumulate)
//   q, k = rotary(y_q, y_k) at each token's absolute position; v = y_v
//
// The projection is a plain GEMM and goes to rocBLAS (bf16 in/out, fp32 compute).  A
// work-group of a few tokens then reads their y rows once, in 16-byte pieces: it finds each
// token's position from cu_q / seq_lens (suffix token i of request r sits at L_r - S_r + i),
// computes the D/2 rotary angles p * theta^(-2i/D) in fp64 (the frequencies once per
// work-group), reduced mod 2 pi before the fp32 sine and cosine, rotates the (i, i + D/2)
// pairs of every query and key head in fp32 and writes bf16 (round to nearest even)
// Q [T][Hq][D], K [T][Hkv][D] and V [T][Hkv][D]; K and V then go to the pool through the KV
// scatter.
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <cmath>
#include <mutex>

#include "../host/internal.hpp"

namespace {

constexpr int kThreads = 256;
constexpr int kTokens = 4;     // tokens per work-group (the rotary frequencies are shared)

typedef uint16_t u16x8_t __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {  // nearest even; inputs finite
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Work-group = kTokens consecutive tokens.  A task is 8 consecutive rotary pairs (i .. i+7,
// i+D/2 .. i+D/2+7) of one head of one token: two 16-byte loads and two 16-byte stores.
template <int D>
__global__ __launch_bounds__(kThreads) void qkv_rope_kernel(
    const uint16_t* __restrict__ y, int64_t n_tokens, int hq, int hkv,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ seq_lens, int n_reqs,
    double theta, uint16_t* __restrict__ q_out, uint16_t* __restrict__ k_out,
    uint16_t* __restrict__ v_out) {
  constexpr int HALF = D / 2;
  constexpr int CH = HALF / 8;                       // 8-pair chunks per head
  __shared__ double freq[HALF];
  __shared__ float cs[kTokens][HALF], sn[kTokens][HALF];
  __shared__ int pos_s[kTokens];
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kTokens;
  const int nt = static_cast<int>(min<int64_t>(kTokens, n_tokens - t0));
  const int tid = threadIdx.x;
  if (tid < nt) {  // request of token t: the last r with cu_q[r] <= t
    const int64_t t = t0 + tid;
    int lo = 0, hi = n_reqs - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) / 2;
      if (cu_q[mid] <= t) lo = mid; else hi = mid - 1;
    }
    pos_s[tid] = seq_lens[lo] - (cu_q[lo + 1] - cu_q[lo]) + static_cast<int>(t - cu_q[lo]);
  }
  for (int i = tid; i < HALF; i += kThreads) freq[i] = std::pow(theta, -2.0 * i / D);
  __syncthreads();
  for (int e = tid; e < nt * HALF; e += kThreads) {
    const int j = e / HALF, i = e % HALF;
    const double a = std::fmod(static_cast<double>(pos_s[j]) * freq[i], 6.283185307179586476925);
    float s, c;
    sincosf(static_cast<float>(a), &s, &c);
    cs[j][i] = c;
    sn[j][i] = s;
  }
  __syncthreads();
  const int nrot = hq + hkv, width = (hq + 2 * hkv) * D;
  for (int e = tid; e < nt * nrot * CH; e += kThreads) {
    const int j = e / (nrot * CH), r = e % (nrot * CH), h = r / CH, i = (r % CH) * 8;
    const int64_t t = t0 + j;
    const uint16_t* src = y + t * width + h * D + i;
    const u16x8_t lo = *reinterpret_cast<const u16x8_t*>(src);
    const u16x8_t hi = *reinterpret_cast<const u16x8_t*>(src + HALF);
    u16x8_t olo, ohi;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float a = bf16_to_f32(lo[k]), b = bf16_to_f32(hi[k]);
      const float c = cs[j][i + k], s = sn[j][i + k];
      olo[k] = f32_to_bf16(a * c - b * s);
      ohi[k] = f32_to_bf16(b * c + a * s);
    }
    uint16_t* dst = h < hq ? q_out + (t * hq + h) * D + i : k_out + (t * hkv + (h - hq)) * D + i;
    *reinterpret_cast<u16x8_t*>(dst) = olo;
    *reinterpret_cast<u16x8_t*>(dst + HALF) = ohi;
  }
  // values: a plain copy of the token's Hkv * D trailing elements of y
  for (int e = tid; e < nt * hkv * (D / 8); e += kThreads) {
    const int j = e / (hkv * (D / 8)), r = e % (hkv * (D / 8));
    const int64_t t = t0 + j;
    *reinterpret_cast<u16x8_t*>(v_out + t * hkv * D + r * 8) =
        *reinterpret_cast<const u16x8_t*>(y + t * width + nrot * D + r * 8);
  }
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
  for (const void* p : {static_cast<const void*>(y_workspace), static_cast<const void*>(q_out),
                        static_cast<const void*>(k_out), static_cast<const void*>(v_out)})
    if (reinterpret_cast<uintptr_t>(p) % 16 != 0)
      return arckv::fail(ARCKV_EINVAL, "qkv_rope: workspace and outputs must be 16-byte aligned");
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
  const dim3 grid(static_cast<unsigned>((n_tokens + kTokens - 1) / kTokens));
  auto* y = static_cast<const uint16_t*>(y_workspace);
  auto* q = static_cast<uint16_t*>(q_out);
  auto* k = static_cast<uint16_t*>(k_out);
  auto* v = static_cast<uint16_t*>(v_out);
  if (head_dim == 64)
    hipLaunchKernelGGL(qkv_rope_kernel<64>, grid, dim3(kThreads), 0, s, y, n_tokens, num_q_heads, num_kv_heads,
                       cu_q, seq_lens, n_reqs, rope_theta, q, k, v);
  else
    hipLaunchKernelGGL(qkv_rope_kernel<128>, grid, dim3(kThreads), 0, s, y, n_tokens, num_q_heads, num_kv_heads,
                       cu_q, seq_lens, n_reqs, rope_theta, q, k, v);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return arckv::fail(ARCKV_EDEVICE, "qkv_rope: %s", hipGetErrorString(e));
  return ARCKV_OK;
}
