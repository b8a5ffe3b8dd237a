// Adam update of exit parameters (Sec. 3 "Tuning": Adam, Kingma and Ba),
// fused over up to kAdamMaxTensors tensors per launch.
//
// Per element, in fp32:
//   m <- b1 m + (1 - b1) g,   v <- b2 v + (1 - b2) g^2,
//   p <- p - (lr / (1 - b1^t)) m / (sqrt(v / (1 - b2^t)) + eps),
// where p is the fp32 master copy when there is one (the stored parameter
// then receives p rounded to its type), else the stored parameter itself.
//
// HBM-bound: per element it reads g, m, v and p and writes m, v, p (and the
// bf16 copy): 30 bytes with an fp32 master and a bf16 parameter.  A block
// owns 4096 consecutive elements of one tensor; each thread issues all 16
// of its 16-byte loads (4 groups of 4 elements) before any arithmetic, so
// every wave keeps its loads in flight together.  The gradient, moment and
// master streams are touched once per update, so their loads and stores
// are non-temporal (14% faster at the 7B output matrix); the parameter,
// which the next step's products read, is stored normally.
#include <hip/hip_runtime.h>

#include "ee_device.h"
#include "launch.h"

namespace ee {

namespace {

constexpr int kAdamThreads = 256;
constexpr int kAdamGroups = 4;  // groups of 4 elements per thread
constexpr int64_t kAdamBlockElems = int64_t{kAdamThreads} * 4 * kAdamGroups;

struct AdamHyper {
  float b1, omb1, b2, omb2, eps, lr_bc1, inv_bc2;
};

__device__ __forceinline__ void adam_elem(const AdamHyper &h, float g, float &m, float &v, float &p) {
  m = h.b1 * m + h.omb1 * g;
  v = h.b2 * v + h.omb2 * (g * g);
  const float denom = sqrtf(v * h.inv_bc2) + h.eps;
  p = p - h.lr_bc1 * (m / denom);
}

template <typename T>
__device__ __forceinline__ f32x4_t load_param4(const T *p);
template <>
__device__ __forceinline__ f32x4_t load_param4<float>(const float *p) {
  return *reinterpret_cast<const f32x4_t *>(p);
}
template <>
__device__ __forceinline__ f32x4_t load_param4<bf16_t>(const bf16_t *p) {
  const u32x2_t u = *reinterpret_cast<const u32x2_t *>(p);
  return f32x4_t{__uint_as_float(u[0] << 16), __uint_as_float(u[0] & 0xFFFF0000u), __uint_as_float(u[1] << 16),
                 __uint_as_float(u[1] & 0xFFFF0000u)};
}
template <typename T>
__device__ __forceinline__ void store_param4(T *p, f32x4_t v);
template <>
__device__ __forceinline__ void store_param4<float>(float *p, f32x4_t v) {
  *reinterpret_cast<f32x4_t *>(p) = v;
}
template <>
__device__ __forceinline__ void store_param4<bf16_t>(bf16_t *p, f32x4_t v) {
  const u32x2_t u = {static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16),
                     static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16)};
  *reinterpret_cast<u32x2_t *>(p) = u;
}

// Full block: kAdamBlockElems elements starting at `base`, all inside the tensor.
template <typename T, bool MASTER>
__device__ __forceinline__ void adam_block_full(const AdamTensorArgs &t, const AdamHyper &h, int64_t base) {
  T *__restrict__ param = static_cast<T *>(t.param);
  float *__restrict__ master = t.master;
  const float *__restrict__ grad = t.grad;
  float *__restrict__ mom1 = t.exp_avg;
  float *__restrict__ mom2 = t.exp_avg_sq;
  f32x4_t g[kAdamGroups], m[kAdamGroups], v[kAdamGroups], p[kAdamGroups];
  static_for<kAdamGroups>([&](auto q) EE_ALWAYS_INLINE {
    const int64_t i = base + (static_cast<int64_t>(decltype(q)::value) * kAdamThreads + threadIdx.x) * 4;
    g[q] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(grad + i));
    m[q] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(mom1 + i));
    v[q] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(mom2 + i));
    if constexpr (MASTER)
      p[q] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(master + i));
    else
      p[q] = load_param4<T>(param + i);
  });
  static_for<kAdamGroups>([&](auto q) EE_ALWAYS_INLINE {
    constexpr int Q = decltype(q)::value;
    const int64_t i = base + (static_cast<int64_t>(Q) * kAdamThreads + threadIdx.x) * 4;
    static_for<4>([&](auto e) EE_ALWAYS_INLINE {
      constexpr int E = decltype(e)::value;
      float mm = m[Q][E], vv = v[Q][E], pp = p[Q][E];
      adam_elem(h, g[Q][E], mm, vv, pp);
      m[Q][E] = mm;
      v[Q][E] = vv;
      p[Q][E] = pp;
    });
    __builtin_nontemporal_store(m[Q], reinterpret_cast<f32x4_t *>(mom1 + i));
    __builtin_nontemporal_store(v[Q], reinterpret_cast<f32x4_t *>(mom2 + i));
    if constexpr (MASTER) __builtin_nontemporal_store(p[Q], reinterpret_cast<f32x4_t *>(master + i));
    store_param4<T>(param + i, p[Q]);
  });
}

// Last, partial block of a tensor: one element per thread per pass.
template <typename T, bool MASTER>
__device__ __forceinline__ void adam_block_tail(const AdamTensorArgs &t, const AdamHyper &h, int64_t base) {
  T *param = static_cast<T *>(t.param);
  for (int64_t i = base + threadIdx.x; i < t.numel; i += kAdamThreads) {
    float m = t.exp_avg[i], v = t.exp_avg_sq[i];
    float p = MASTER ? t.master[i] : to_f32(param[i]);
    adam_elem(h, t.grad[i], m, v, p);
    t.exp_avg[i] = m;
    t.exp_avg_sq[i] = v;
    if constexpr (MASTER) t.master[i] = p;
    param[i] = from_f32<T>(p);
  }
}

template <typename T, bool MASTER>
__device__ __forceinline__ void adam_block(const AdamTensorArgs &t, const AdamHyper &h, int64_t base) {
  if (base + kAdamBlockElems <= t.numel)
    adam_block_full<T, MASTER>(t, h, base);
  else
    adam_block_tail<T, MASTER>(t, h, base);
}

__global__ __launch_bounds__(kAdamThreads) void adam_kernel(AdamBatchArgs b) {
  int k = 0;
  for (int i = 1; i < b.count; ++i)
    if (static_cast<int64_t>(blockIdx.x) >= b.t[i].first_block) k = i;
  const AdamTensorArgs t = b.t[k];
  const int64_t base = (static_cast<int64_t>(blockIdx.x) - t.first_block) * kAdamBlockElems;
  const AdamHyper h{b.beta1, 1.0f - b.beta1, b.beta2, 1.0f - b.beta2, b.eps, b.lr_bc1, b.inv_bc2};
  const bool master = t.master != nullptr;
  if (t.bf16) {
    if (master)
      adam_block<bf16_t, true>(t, h, base);
    else
      adam_block<bf16_t, false>(t, h, base);
  } else {
    if (master)
      adam_block<float, true>(t, h, base);
    else
      adam_block<float, false>(t, h, base);
  }
}

}  // namespace

int64_t adam_blocks(int64_t numel) { return (numel + kAdamBlockElems - 1) / kAdamBlockElems; }

hipError_t launch_adam(AdamBatchArgs b, hipStream_t stream) {
  int64_t blocks = 0;
  for (int i = 0; i < b.count; ++i) {
    b.t[i].first_block = blocks;
    blocks += adam_blocks(b.t[i].numel);
  }
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(adam_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kAdamThreads), 0, stream, b);
  return hipGetLastError();
}

}  // namespace ee
