// Localized group construction and the group-relative policy-loss factors
// (Sec. 3.3 and Sec. 4.1):
//
//  * allocate_kernel: each root's continuation slots are assigned to its
//    retained branch points in rank order (the default 3 + 4 for two points
//    per root); slots of a point that was not retained go to the root's best
//    point, so a root with one valid point still fills all of its slots; a
//    root with none branches at a fallback position.
//  * advantages_kernel: the mean-centred group advantage A_j = R_j - mean(R)
//    without standard-deviation normalisation.
//  * policy_grad_kernel: per token, the derivative of the asymmetrically
//    clipped surrogate -min(r A, clip(r, 1 - eps_low, 1 + eps_high) A) with
//    respect to log pi (r = pi / pi_old), times the token-level aggregation
//    factor; tokens before their trajectory's branch point (the reused
//    prefix of a continuation) and tokens outside the loss mask contribute
//    nothing.  The result is the per-token g that the lm-head backward pass
//    takes.
#include "hdl_internal.h"

namespace hdl {
namespace {

constexpr int kMaxAlloc = 16;

struct Alloc {
  int32_t n[kMaxAlloc];
};

__global__ __launch_bounds__(256) void allocate_kernel(const int32_t* __restrict__ idx,
                                                       const int32_t* __restrict__ count, int64_t n_roots,
                                                       int k, Alloc alloc, int total, int32_t fallback,
                                                       int32_t* __restrict__ branch_pos,
                                                       int32_t* __restrict__ branch_rank) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= n_roots) return;
  int c = count[r];
  c = c < 0 ? 0 : (c > k ? k : c);
  int32_t* pos = branch_pos + r * total;
  int32_t* rnk = branch_rank ? branch_rank + r * total : nullptr;
  int slot = 0;
  for (int j = 0; j < k; ++j) {
    const int target = j < c ? j : 0;
    const int32_t p = c > 0 ? idx[r * k + target] : fallback;
    for (int u = 0; u < alloc.n[j]; ++u, ++slot) {
      pos[slot] = p;
      if (rnk) rnk[slot] = c > 0 ? target : -1;
    }
  }
}

// One workgroup per group; the mean is a fixed-order tree sum.
__global__ __launch_bounds__(256) void advantages_kernel(const float* __restrict__ rewards, int group_size,
                                                         float* __restrict__ adv) {
  __shared__ float part[256];
  const int64_t g = blockIdx.x;
  const float* R = rewards + g * group_size;
  float s = 0.f;
  for (int j = threadIdx.x; j < group_size; j += 256) s += R[j];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  const float mean = part[0] / static_cast<float>(group_size);
  for (int j = threadIdx.x; j < group_size; j += 256) adv[g * group_size + j] = R[j] - mean;
}

struct PolicyGradArgs {
  const float* adv;
  const int32_t* traj;
  const int32_t* pos;
  const int32_t* start;
  const float* logp_new;
  const float* logp_old;
  const uint8_t* loss_mask;
  int64_t n_tokens, n_traj;
  float eps_low, eps_high, scale;   // scale <= 0: 1 / max(1, *n_trained)
  float* grad;
  float* loss;
  unsigned long long* n_trained;    // trained-token count (device), or nullptr
};

// Whether the loss trains on a token: in the loss mask, of a known
// trajectory, and (with positions) at or after the trajectory's first
// trained position -- a continuation trains only its suffix.
__device__ __forceinline__ bool trained(const PolicyGradArgs& p, int32_t j, int32_t pos, uint8_t m) {
  bool on = m != 0 && j >= 0 && j < p.n_traj;
  if (p.pos && p.start) on = on && pos >= p.start[j];
  return on;
}

// The aggregation factor of this call: the caller's scale, or the
// token-level mean over the trained tokens counted by count_trained_kernel.
__device__ __forceinline__ float call_scale(const PolicyGradArgs& p) {
  if (p.scale > 0.f) return p.scale;
  const unsigned long long n = *p.n_trained;
  return static_cast<float>(1.0 / static_cast<double>(n > 0 ? n : 1));
}

// One token's factor; m is the token's loss-mask byte (1 when there is no
// mask), sc the call's aggregation factor.
__device__ __forceinline__ void token_factor(const PolicyGradArgs& p, float sc, int32_t j, int32_t pos, uint8_t m,
                                             float ln, float lo, float& gv, float& lv) {
  const bool on = trained(p, j, pos, m);
  gv = 0.f;
  lv = 0.f;
  if (on) {
    const float a = p.adv[j];
    const float r = expf(ln - lo);
    const float rc = fminf(fmaxf(r, 1.f - p.eps_low), 1.f + p.eps_high);
    const float unclipped = r * a, clipped = rc * a;
    // d/dlog pi of min(r A, clip(r) A): r A where the unclipped term is the
    // minimum (ties included), 0 where the clipped constant is
    gv = unclipped <= clipped ? -a * r * sc : 0.f;
    lv = -fminf(unclipped, clipped) * sc;
  }
}

// VEC = 4: four consecutive tokens per thread through 16-byte loads and
// stores (every per-token array 16-byte aligned, the mask 4-byte aligned);
// VEC = 1: one token per thread, any alignment.
template <int VEC>
__global__ __launch_bounds__(256) void policy_grad_kernel(PolicyGradArgs p) {
  const int64_t n0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * VEC;
  if (n0 >= p.n_tokens) return;
  const float sc = call_scale(p);
  if (VEC == 4 && n0 + 4 <= p.n_tokens) {
    const int4 j = *reinterpret_cast<const int4*>(p.traj + n0);
    const int4 ps = p.pos ? *reinterpret_cast<const int4*>(p.pos + n0) : make_int4(0, 0, 0, 0);
    const float4 ln = *reinterpret_cast<const float4*>(p.logp_new + n0);
    const float4 lo = *reinterpret_cast<const float4*>(p.logp_old + n0);
    const uchar4 m = p.loss_mask ? *reinterpret_cast<const uchar4*>(p.loss_mask + n0) : make_uchar4(1, 1, 1, 1);
    float4 g, l;
    token_factor(p, sc, j.x, ps.x, m.x, ln.x, lo.x, g.x, l.x);
    token_factor(p, sc, j.y, ps.y, m.y, ln.y, lo.y, g.y, l.y);
    token_factor(p, sc, j.z, ps.z, m.z, ln.z, lo.z, g.z, l.z);
    token_factor(p, sc, j.w, ps.w, m.w, ln.w, lo.w, g.w, l.w);
    *reinterpret_cast<float4*>(p.grad + n0) = g;
    if (p.loss) *reinterpret_cast<float4*>(p.loss + n0) = l;
    return;
  }
  const int64_t n1 = n0 + VEC < p.n_tokens ? n0 + VEC : p.n_tokens;
  for (int64_t n = n0; n < n1; ++n) {
    float gv, lv;
    token_factor(p, sc, p.traj[n], p.pos ? p.pos[n] : 0, p.loss_mask ? p.loss_mask[n] : 1, p.logp_new[n],
                 p.logp_old[n], gv, lv);
    p.grad[n] = gv;
    if (p.loss) p.loss[n] = lv;
  }
}

__global__ void clear_count_kernel(unsigned long long* n) { *n = 0ull; }

// Trained tokens of the call: a grid-stride loop over VEC tokens at a time
// (VEC = 4 under the alignment policy_grad_kernel's vector path needs), then
// one integer atomic add per workgroup -- exact, so the order does not
// matter, and few enough workgroups that the adds to one address do not
// queue up.  1024-thread workgroups keep 32 waves per CU loading with only
// 512 atomics.
constexpr int kCountBlocks = 512;
constexpr int kCountThreads = 1024;

template <int VEC>
__global__ __launch_bounds__(kCountThreads) void count_trained_kernel(PolicyGradArgs p) {
  unsigned c = 0;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x * VEC;
  for (int64_t n0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * VEC; n0 < p.n_tokens;
       n0 += stride) {
    if (VEC == 4 && n0 + 4 <= p.n_tokens) {
      const int4 j = *reinterpret_cast<const int4*>(p.traj + n0);
      const int4 ps = p.pos ? *reinterpret_cast<const int4*>(p.pos + n0) : make_int4(0, 0, 0, 0);
      const uchar4 m = p.loss_mask ? *reinterpret_cast<const uchar4*>(p.loss_mask + n0) : make_uchar4(1, 1, 1, 1);
      c += trained(p, j.x, ps.x, m.x) + trained(p, j.y, ps.y, m.y) + trained(p, j.z, ps.z, m.z) +
           trained(p, j.w, ps.w, m.w);
    } else {
      const int64_t n1 = n0 + VEC < p.n_tokens ? n0 + VEC : p.n_tokens;
      for (int64_t n = n0; n < n1; ++n)
        c += trained(p, p.traj[n], p.pos ? p.pos[n] : 0, p.loss_mask ? p.loss_mask[n] : 1);
    }
  }
  __shared__ unsigned part[kCountThreads / 64];
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long t = 0;
    for (int w = 0; w < kCountThreads / 64; ++w) t += part[w];
    if (t) atomicAdd(p.n_trained, t);
  }
}

}  // namespace

hipError_t launch_allocate(const int32_t* idx, const int32_t* count, int64_t n_roots, int k,
                           const int32_t* alloc, int total, int32_t fallback, int32_t* branch_pos,
                           int32_t* branch_rank, hipStream_t stream) {
  Alloc a{};
  for (int j = 0; j < k && j < kMaxAlloc; ++j) a.n[j] = alloc[j];
  const int64_t blocks = (n_roots + 255) / 256;
  hipLaunchKernelGGL(allocate_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, idx, count,
                     n_roots, k, a, total, fallback, branch_pos, branch_rank);
  return hipGetLastError();
}

hipError_t launch_advantages(const float* rewards, int64_t n_groups, int group_size, float* adv,
                             hipStream_t stream) {
  hipLaunchKernelGGL(advantages_kernel, dim3(static_cast<unsigned>(n_groups)), dim3(256), 0, stream, rewards,
                     group_size, adv);
  return hipGetLastError();
}

hipError_t launch_policy_grad(const float* adv, const int32_t* traj, const int32_t* pos, const int32_t* start,
                              const float* logp_new, const float* logp_old, const uint8_t* loss_mask,
                              int64_t n_tokens, int64_t n_traj, float eps_low, float eps_high, float scale,
                              float* grad, float* loss, int64_t* n_trained, hipStream_t stream) {
  const PolicyGradArgs a{adv, traj, pos, start, logp_new, logp_old, loss_mask, n_tokens, n_traj,
                         eps_low, eps_high, scale, grad, loss,
                         reinterpret_cast<unsigned long long*>(n_trained)};
  auto al = [](const void* q, uintptr_t b) { return q == nullptr || reinterpret_cast<uintptr_t>(q) % b == 0; };
  const bool vec = al(traj, 16) && al(pos, 16) && al(logp_new, 16) && al(logp_old, 16) && al(grad, 16) &&
                   al(loss, 16) && al(loss_mask, 4);
  const int64_t blocks = vec ? (n_tokens + 1023) / 1024 : (n_tokens + 255) / 256;
  if (n_trained) {
    hipLaunchKernelGGL(clear_count_kernel, dim3(1), dim3(1), 0, stream, a.n_trained);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t per_block = static_cast<int64_t>(kCountThreads) * (vec ? 4 : 1);
    const int64_t need = (n_tokens + per_block - 1) / per_block;
    const unsigned cb = static_cast<unsigned>(need < kCountBlocks ? need : kCountBlocks);
    if (vec)
      hipLaunchKernelGGL(count_trained_kernel<4>, dim3(cb), dim3(kCountThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(count_trained_kernel<1>, dim3(cb), dim3(kCountThreads), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (vec)
    hipLaunchKernelGGL(policy_grad_kernel<4>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(policy_grad_kernel<1>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace hdl
