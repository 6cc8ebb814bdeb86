// Reuse criterion and next-window selection (Sec. 3.1) and the fallback
// statistics of App. E, after acceptance.
//
// Per sequence, the corrected prefix Pi+ = (accepted tokens, correction) is
// looked up among the root-to-depth-tau paths of the hypothesis tree T_t
// (tau = A + 1): a wave gives every lane a few candidate nodes at depth tau
// and each walks its parents, comparing tokens with Pi+ from the end; the
// smallest matching node wins. The overlap mass Omega_k at the root row is
// the final head's probability mass on the early-exit top-k ids, summed in
// fp64 in id-rank order. One workgroup serves the whole batch so that the
// running statistics are accumulated in sequence order, without atomics.
#include "kernels.h"
#include "msd.h"

namespace msd {
namespace {

constexpr int kWaves = 4;

__global__ __launch_bounds__(64 * kWaves) void reuse_kernel(ReuseArgs a) {
  __shared__ int16_t parent[kMaxTreeNodes];
  __shared__ uint8_t depth[kMaxTreeNodes];
  __shared__ int32_t pre[kWaves][kMaxSlots + 1];   // Pi+ per wave, depth 1..tau
  __shared__ int32_t fb[kMaxSlots * kWaves];       // per-sequence results for the statistics
  __shared__ double om[kMaxSlots * kWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = a.tree.n_nodes;
  for (int i = tid; i < n; i += blockDim.x) {
    parent[i] = a.tree.parent[i];
    depth[i] = a.tree.depth[i];
  }
  __syncthreads();
  const bool with_omega = a.logits && a.lse && a.ee_ids;
  double om_sum = 0.0;
  uint64_t n_fb = 0, n_fb1 = 0;
  for (int b0 = 0; b0 < a.batch; b0 += kMaxSlots * kWaves) {
    for (int bb = wave; bb < kMaxSlots * kWaves && b0 + bb < a.batch; bb += kWaves) {
      const int b = b0 + bb;
      int A = a.acc_len[b];
      A = A < 0 ? 0 : (A > a.n_slots - 1 ? a.n_slots - 1 : A);
      const int tau = A + 1;
      // Pi+ at depths 1..tau: the accepted slots' tokens, then the correction
      for (int r = 1 + lane; r <= tau; r += 64) {
        int tok;
        if (r <= A) {
          int slot = a.path[(size_t)b * a.n_slots + r];
          slot = slot < 0 ? 0 : (slot >= a.n_slots ? a.n_slots - 1 : slot);
          tok = a.tokens[(size_t)b * a.n_slots + slot];
        } else {
          tok = a.next_tok[b];
        }
        pre[wave][r] = tok;
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const int32_t* tt = a.tree_tokens + (size_t)b * n;
      int best = 0x7fffffff;
      for (int v = lane; v < n; v += 64) {
        if (depth[v] != tau) continue;
        int u = v, r = tau;
        bool ok = true;
        while (u >= 0 && ok) {
          ok = tt[u] == pre[wave][r];
          u = parent[u];
          --r;
        }
        if (ok && r == 0 && v < best) best = v;
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const int other = __shfl_xor(best, o);
        best = other < best ? other : best;
      }
      const bool found = best != 0x7fffffff;
      double omega = 0.0;
      if (with_omega) {
        const size_t m0 = (size_t)b * a.n_slots;  // the root row predicts position t + 1
        const double l = (double)a.lse[m0];
        double p = 0.0;
        if (lane < a.kappa) {
          int id = a.ee_ids[m0 * a.kappa + lane];
          id = id < 0 ? 0 : (id >= a.vocab ? a.vocab - 1 : id);
          p = exp((double)a.logits[m0 * a.vocab + id] - l);
        }
        // a fixed-shape tree over the lanes (lane 0 ends with the sum)
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) p += __shfl_down(p, o);
        omega = __shfl(p, 0);
      }
      if (lane == 0) {
        a.next_case[b] = found ? (A == 0 ? MSD_NEXT_BRANCH : MSD_NEXT_CONTINUE) : MSD_NEXT_FRESH;
        a.next_node[b] = found ? best : -1;
        if (with_omega && a.omega) a.omega[b] = (float)omega;
        fb[bb] = found ? 0 : (A == 0 ? 2 : 1);
        om[bb] = omega;
      }
    }
    __syncthreads();
    if (tid == 0) {
      for (int bb = 0; bb < kMaxSlots * kWaves && b0 + bb < a.batch; ++bb) {
        n_fb += fb[bb] != 0;
        n_fb1 += fb[bb] == 2;
        om_sum += om[bb];
      }
    }
    __syncthreads();
  }
  if (tid == 0 && a.stats) {
    a.stats->trials += (uint64_t)a.batch;
    a.stats->fallbacks += n_fb;
    a.stats->fallbacks_tau1 += n_fb1;
    if (with_omega) {
      a.stats->omega_trials += (uint64_t)a.batch;
      a.stats->omega_sum += om_sum;
    }
  }
}

}  // namespace

hipError_t launch_reuse(const ReuseArgs& a, hipStream_t s) {
  if (a.batch < 1 || a.tree.n_nodes < 1 || a.tree.n_nodes > kMaxTreeNodes || a.n_slots < 1 ||
      a.n_slots > kMaxSlots || (a.logits && (a.kappa < 1 || a.kappa > 64)))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(reuse_kernel, dim3(1), dim3(64 * kWaves), 0, s, a);
  return hipGetLastError();
}

}  // namespace msd
