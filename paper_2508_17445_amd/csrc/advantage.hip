// TreePO advantage over the rollout tree (TreePO Sec. 2.3, Eq. groups and
// Eq. tree_ae; the sub-group-size weighted variant Eq. tree_ae_sgw of
// Sec. 4.2), one workgroup, fp64 arithmetic:
//   1. every sub-group's mean reward, and whether its rewards are all equal
//      (a query whose group is all equal is rejected);
//   2. every kept position's sub-group advantages R_p - mean(G_a) over its
//      strict predecessors a, pooled by their mean (or |G_a|-weighted mean),
//      and the sums of all of them and of their squares;
//   3. one global population standard deviation; advantage = pooled / std.
// Sums run in a fixed order (per-thread partials in index order, then a
// fixed tree), so results do not depend on scheduling.  The work is a few
// thousand sub-groups and pairs per batch: a latency-bound kernel.
#include "kernels.h"

#include <math.h>

namespace treepo {
namespace {

constexpr int kAdvThreads = 1024;
// Rewards of up to this many positions are staged in LDS first, so that the
// member loops' reads are LDS reads instead of dependent global loads.
constexpr int kAdvLdsRewards = 8192;

__global__ __launch_bounds__(kAdvThreads) void advantage_kernel(AdvantageArgs a) {
  __shared__ double red_s1[kAdvThreads];
  __shared__ double red_s2[kAdvThreads];
  __shared__ int32_t red_n[kAdvThreads];
  __shared__ float rew[kAdvLdsRewards];
  const int tid = threadIdx.x;
  const bool staged = a.n_pos <= kAdvLdsRewards;
  if (staged) {
    for (int p = tid; p < a.n_pos; p += kAdvThreads) rew[p] = a.rewards[p];
    __syncthreads();
  }
  const float* R = staged ? rew : a.rewards;

  // 1. sub-group means and the all-equal test
  for (int g = tid; g < a.n_groups; g += kAdvThreads) {
    const int b = a.grp_off[g], e = a.grp_off[g + 1];
    double sum = 0.0;
    float lo = INFINITY, hi = -INFINITY;
    for (int k = b; k < e; ++k) {
      const float r = R[a.grp_mem[k]];
      sum += static_cast<double>(r);
      lo = fminf(lo, r);
      hi = fmaxf(hi, r);
    }
    a.gmean[g] = e > b ? sum / static_cast<double>(e - b) : 0.0;
    a.gkeep[g] = hi != lo;
  }
  __syncthreads();

  // 2. pooled sub-group advantages of kept positions; global sums
  double s1 = 0.0, s2 = 0.0;
  int32_t cnt = 0;
  for (int p = tid; p < a.n_pos; p += kAdvThreads) {
    const int b = a.pos_off[p], e = a.pos_off[p + 1];
    double pooled = 0.0;
    if (a.gkeep[a.pos_root[p]] && e > b) {
      const double r = static_cast<double>(R[p]);
      double num = 0.0, den = 0.0;
      for (int k = b; k < e; ++k) {
        const int g = a.pos_grp[k];
        const double d = r - a.gmean[g];
        const double w = a.size_weighted ? static_cast<double>(a.grp_off[g + 1] - a.grp_off[g]) : 1.0;
        num += w * d;
        den += w;
        s1 += d;
        s2 += d * d;
        ++cnt;
      }
      pooled = num / den;
    }
    a.pooled[p] = pooled;
  }
  red_s1[tid] = s1;
  red_s2[tid] = s2;
  red_n[tid] = cnt;
  __syncthreads();
  for (int w = kAdvThreads / 2; w > 0; w >>= 1) {
    if (tid < w) {
      red_s1[tid] += red_s1[tid + w];
      red_s2[tid] += red_s2[tid + w];
      red_n[tid] += red_n[tid + w];
    }
    __syncthreads();
  }

  // 3. divide by the global population standard deviation
  const int32_t n = red_n[0];
  double sigma = 0.0;
  if (n > 0) {
    const double m = red_s1[0] / n;
    const double var = red_s2[0] / n - m * m;
    sigma = var > 0.0 ? sqrt(var) : 0.0;
  }
  for (int p = tid; p < a.n_pos; p += kAdvThreads) {
    const int b = a.pos_off[p], e = a.pos_off[p + 1];
    const bool kept = a.gkeep[a.pos_root[p]] && e > b;
    a.adv[p] = kept && sigma > 0.0 ? static_cast<float>(a.pooled[p] / sigma) : 0.f;
  }
}

}  // namespace

hipError_t launch_advantage(const AdvantageArgs& a, hipStream_t s) {
  if (a.n_pos <= 0) return hipSuccess;
  hipLaunchKernelGGL(advantage_kernel, dim3(1), dim3(kAdvThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace treepo
