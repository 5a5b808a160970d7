// Fingerprint reduction and the dual-metric gate (Section 2.3-2.5).
//
//   fp_colsum   : one read of the block input x; partial column sums over
//                 16-row chunks that never straddle a camera (HBM-bound).
//   fp_compare  : per 32-column slice: finishes each camera's token mean
//                 (global channel), gathers the spatial fingerprint rows,
//                 accumulates the per-group partial terms of Eq. 5-6 against
//                 the previous generation's fingerprint and overwrites it with
//                 the current one (the fingerprint cache is refreshed at every
//                 evaluation, computed or skipped).
//   gate_decide : one workgroup; reduces the partial terms in a fixed order
//                 (deterministic), forms s = min-cosine and d = max-deviation,
//                 applies the adaptive threshold (Eq. 8-9), the skip rule
//                 (Eq. 7), the staleness bound, and writes the block's skip
//                 flag, its staleness counter and the statistics.
//
// Fingerprint storage for one (t, b): [n_srows + n_cams][C] float -- the
// spatial rows in group order, then one token-mean row per camera.
#include "xc_internal.h"

#include <math.h>

namespace xc {

namespace {

constexpr int kRec = kFpRecord;  // dot_s, nn_s, pp_s, maxabs_s, sumabs_prev_s, dot_g, nn_g, pp_g

__global__ __launch_bounds__(1024) void fp_colsum_kernel(const float* __restrict__ x, int C, const int4* __restrict__ chunks,
                                                          float* __restrict__ partial) {
  const int4 ch = chunks[blockIdx.x];
  const int C4 = C >> 2;
  const float4* base = reinterpret_cast<const float4*>(x + (long long)ch.x * C);
  float4* out = reinterpret_cast<float4*>(partial + (long long)blockIdx.x * C);
  for (int c4 = threadIdx.x; c4 < C4; c4 += blockDim.x) {
    float4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int r = 0; r < ch.y; ++r) {
      float4 v = base[(long long)r * C4 + c4];
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
    out[c4] = acc;
  }
}

__device__ __forceinline__ double block_reduce(double v, double* s_red, bool is_max) {
  // 256 threads: wave reduction, then across the 4 waves through LDS.
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    double o = __shfl_xor(v, off, 64);
    v = is_max ? fmax(v, o) : v + o;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  double r = s_red[0];
  for (int w = 1; w < 4; ++w) r = is_max ? fmax(r, s_red[w]) : r + s_red[w];
  return r;
}

__global__ __launch_bounds__(256) void fp_compare_kernel(const float* __restrict__ x, int C, FpTables t,
                                                         const float* __restrict__ partial,
                                                         float* __restrict__ fp_prev, double* __restrict__ records) {
  __shared__ double s_red[4];
  const int cl = threadIdx.x % kFpCompareCols;
  const int rl = threadIdx.x / kFpCompareCols;
  constexpr int kRowLanes = 256 / kFpCompareCols;
  const int c = blockIdx.x * kFpCompareCols + cl;
  const bool col_ok = c < C;
  for (int g = 0; g < t.n_groups; ++g) {
    double acc[kRec] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (col_ok) {
      for (int i = t.grp_srow_begin[g] + rl; i < t.grp_srow_begin[g + 1]; i += kRowLanes) {
        double cur = (double)x[(long long)t.srows[i] * C + c];
        float* pp = fp_prev + (long long)i * C + c;
        double prev = (double)*pp;
        acc[0] += cur * prev;
        acc[1] += cur * cur;
        acc[2] += prev * prev;
        acc[3] = fmax(acc[3], fabs(cur - prev));
        acc[4] += fabs(prev);
        *pp = (float)cur;
      }
      for (int v = t.grp_cam_begin[g] + rl; v < t.grp_cam_begin[g + 1]; v += kRowLanes) {
        double s = 0.0;
        for (int k = t.cam_chunk_begin[v]; k < t.cam_chunk_begin[v + 1]; ++k) s += (double)partial[(long long)k * C + c];
        float mean = (float)(s / (double)t.cam_tokens[v]);
        double cur = (double)mean;
        float* pp = fp_prev + (long long)(t.n_srows + v) * C + c;
        double prev = (double)*pp;
        acc[5] += cur * prev;
        acc[6] += cur * cur;
        acc[7] += prev * prev;
        *pp = mean;
      }
    }
    double* rec = records + ((long long)blockIdx.x * kMaxGroups + g) * kRec;
#pragma unroll
    for (int k = 0; k < kRec; ++k) {
      double r = block_reduce(acc[k], s_red, k == 3);
      if (threadIdx.x == 0) rec[k] = r;
    }
  }
}

__device__ __forceinline__ double cos_from(double dot, double nn, double pp) {
  double den = sqrt(nn) * sqrt(pp);
  return dot / fmax(den, 1e-12);
}

// One wave.  evaluate == 0: the block is computed without a test (warmup,
// forced pass, step-0 force, first visit): clear the flag and the staleness.
__global__ void gate_decide_kernel(const double* __restrict__ records, int n_wg, GateArgs ga, GateState gs,
                                   int sb, int b, int evaluate) {
  const int lane = threadIdx.x;
  if (!evaluate) {
    if (lane == 0) {
      gs.flags[b] = 0;
      gs.stale[sb] = 0;
    }
    return;
  }
  double s_min = 1e300, d_max = -1e300;
  for (int g = 0; g < ga.n_groups; ++g) {
    double tot[kRec];
    for (int k = 0; k < kRec; ++k) {
      // lanes stride the workgroup records; a fixed-shape tree keeps the sum deterministic
      double v = 0.0;
      for (int w = lane; w < n_wg; w += 64) {
        double r = records[((long long)w * kMaxGroups + g) * kRec + k];
        v = (k == 3) ? fmax(v, r) : v + r;
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        double o = __shfl_xor(v, off, 64);
        v = (k == 3) ? fmax(v, o) : v + o;
      }
      tot[k] = v;
    }
    double cs = cos_from(tot[0], tot[1], tot[2]);
    double cg = cos_from(tot[5], tot[6], tot[7]);
    double mean_prev = tot[4] / (double)ga.spatial_count[g];
    double dg = tot[3] / (mean_prev + (double)ga.eps);
    s_min = fmin(s_min, fmin(cs, cg));
    d_max = fmax(d_max, dg);
  }
  if (ga.action_dim > 0) {
    double dot = 0, nn = 0, pp = 0;
    for (int i = 0; i < ga.action_dim; ++i) {
      double a = ga.action[i], p = ga.action_prev[i];
      dot += a * p;
      nn += a * a;
      pp += p * p;
    }
    s_min = fmin(s_min, cos_from(dot, nn, pp));
  }
  if (lane != 0) return;
  double ema = (double)gs.ema[sb];
  const bool has_ema = !isnan(ema);
  double tau;
  if (ga.adaptive)
    tau = has_ema ? fmax((double)ga.tau_floor, ema - (double)ga.margin) : (double)ga.tau_floor;
  else
    tau = (double)ga.tau_cos_fixed;
  if (ga.strict0) tau = fmax(tau, (double)ga.tau_strict0);
  if (ga.adaptive) {
    double e = has_ema ? (double)ga.alpha * s_min + (1.0 - (double)ga.alpha) * ema : s_min;
    gs.ema[sb] = (float)e;
  }
  const int stale = gs.stale[sb];
  const bool skip = (s_min >= tau) && (d_max < (double)ga.tau_dev) && (ga.max_stale == 0 || stale < ga.max_stale);
  gs.flags[b] = skip ? 1 : 0;
  gs.stale[sb] = skip ? stale + 1 : 0;
  if (skip) gs.skip_counts[sb] += 1;
  gs.rec_dec[b] = skip ? 1 : 0;
  gs.rec_s[b] = (float)s_min;
  gs.rec_d[b] = (float)d_max;
  gs.rec_tau[b] = (float)tau;
}

}  // namespace

void launch_fp_colsum(const float* x, int C, const FpTables& t, float* partial, hipStream_t st) {
  int threads = ((C / 4 + 63) / 64) * 64;
  if (threads > 1024) threads = 1024;
  fp_colsum_kernel<<<t.n_chunks, threads, 0, st>>>(x, C, t.chunks, partial);
}

int fp_compare_groups_of_wg(int C) { return (C + kFpCompareCols - 1) / kFpCompareCols; }

void launch_fp_compare(const float* x, int C, const FpTables& t, const float* partial, float* fp_prev,
                       double* records, hipStream_t st) {
  fp_compare_kernel<<<fp_compare_groups_of_wg(C), 256, 0, st>>>(x, C, t, partial, fp_prev, records);
}

void launch_gate_decide(const double* records, int n_wg, const GateArgs& ga, const GateState& gs, int sb, int b,
                        int n_blocks, int evaluate, hipStream_t st) {
  (void)n_blocks;
  gate_decide_kernel<<<1, 64, 0, st>>>(records, n_wg, ga, gs, sb, b, evaluate);
}

}  // namespace xc
