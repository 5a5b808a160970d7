// Fingerprint reduction and the dual-metric gate (Section 2.3-2.5).
//
//   fp_colsum   : one read of the block input x; partial column sums over
//                 16-row chunks that never straddle a camera (HBM-bound).
//   fp_compare  : per 32-column slice, one workgroup for the spatial
//                 fingerprint rows and one per camera for its token mean
//                 (global channel); accumulates the per-group partial terms of
//                 Eq. 5-6 against the previous generation's fingerprint and
//                 overwrites it with the current one (the fingerprint cache is
//                 refreshed at every evaluation, computed or skipped).
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

// Block reduction of NF fields at once (256 threads): the per-field
// shuffle chains are independent, so their latencies overlap; one LDS
// exchange across the 4 waves.  Field `max_field` takes the maximum, the
// others the sum; fixed order throughout.
template <int NF>
__device__ __forceinline__ void block_reduce_n(double (&v)[NF], double* s_red, int max_field) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1)
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const double o = __shfl_xor(v[f], off, 64);
      v[f] = f == max_field ? fmax(v[f], o) : v[f] + o;
    }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0)
#pragma unroll
    for (int f = 0; f < NF; ++f) s_red[wave * NF + f] = v[f];
  __syncthreads();
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    double r = s_red[f];
    for (int w = 1; w < 4; ++w) r = f == max_field ? fmax(r, s_red[w * NF + f]) : r + s_red[w * NF + f];
    v[f] = r;
  }
}

// Grid (column slices of 32, spatial row chunks + cameras).  Row y < n_sp
// handles spatial fingerprint rows [16 y, 16 y + 16) (two per lane); row
// y = n_sp + v finishes camera v's token mean from its partial column sums:
// the 8 lanes of a column each sum every 8th chunk (loads issued 4 at a
// time), and the 8 lane sums are combined in lane order through LDS.  Every
// workgroup writes one record per group (zeros for terms it does not own); the
// decision kernel sums the records in a fixed order, so the result is
// deterministic.
constexpr int kSpRows = 2 * (256 / kFpCompareCols);  // spatial rows per workgroup

__global__ __launch_bounds__(256) void fp_compare_kernel(const float* __restrict__ x, int C, FpTables t,
                                                         const float* __restrict__ partial, float* fp0, float* fp1,
                                                         const int* __restrict__ sel, double* __restrict__ records) {
  // cached fingerprint and where the current one goes
  const bool flip = sel != nullptr && *sel != 0;
  const float* fp_prev = flip ? fp1 : fp0;
  float* fp_cur = sel == nullptr ? fp0 : (flip ? fp0 : fp1);
  __shared__ double s_red[4 * 5];
  __shared__ double s_cam[kFpCompareCols][256 / kFpCompareCols + 1];
  const int cl = threadIdx.x % kFpCompareCols;
  const int rl = threadIdx.x / kFpCompareCols;
  constexpr int kRowLanes = 256 / kFpCompareCols;
  const int c = blockIdx.x * kFpCompareCols + cl;
  const bool col_ok = c < C;
  const int wg = blockIdx.y * gridDim.x + blockIdx.x;
  const int n_sp = (t.n_srows + kSpRows - 1) / kSpRows;
  if ((int)blockIdx.y < n_sp) {
    const int i0 = blockIdx.y * kSpRows;
    const int i1 = min(i0 + kSpRows, t.n_srows);
    // this lane's two rows: loads first, then the terms
    const int ia = i0 + rl, ib = i0 + kRowLanes + rl;
    float cur[2] = {0.f, 0.f}, prev[2] = {0.f, 0.f};
    if (col_ok) {
      if (ia < i1) {
        cur[0] = x[(long long)t.srows[ia] * C + c];
        prev[0] = fp_prev[(long long)ia * C + c];
      }
      if (ib < i1) {
        cur[1] = x[(long long)t.srows[ib] * C + c];
        prev[1] = fp_prev[(long long)ib * C + c];
      }
      if (ia < i1) fp_cur[(long long)ia * C + c] = cur[0];
      if (ib < i1) fp_cur[(long long)ib * C + c] = cur[1];
    }
    for (int g = 0; g < t.n_groups; ++g) {
      double* rec = records + ((long long)wg * kMaxGroups + g) * kRec;
      const int gb = t.grp_srow_begin[g], ge = t.grp_srow_begin[g + 1];
      if (ge <= i0 || gb >= i1) {  // no row of this chunk in group g
        if (threadIdx.x < kRec) rec[threadIdx.x] = 0.0;
        continue;
      }
      double acc[5] = {0, 0, 0, 0, 0};
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int i = u == 0 ? ia : ib;
        if (col_ok && i < i1 && i >= gb && i < ge) {
          const double cu = (double)cur[u], pr = (double)prev[u];
          acc[0] += cu * pr;
          acc[1] += cu * cu;
          acc[2] += pr * pr;
          acc[3] = fmax(acc[3], fabs(cu - pr));
          acc[4] += fabs(pr);
        }
      }
      block_reduce_n<5>(acc, s_red, 3);
      if (threadIdx.x == 0)
#pragma unroll
        for (int k = 0; k < kRec; ++k) rec[k] = k < 5 ? acc[k < 5 ? k : 0] : 0.0;
    }
    return;
  }
  const int v = blockIdx.y - n_sp;
  int gv = 0;
  while (gv + 1 < t.n_groups && t.grp_cam_begin[gv + 1] <= v) ++gv;
  double s = 0.0;
  if (col_ok) {
    const int k0 = t.cam_chunk_begin[v], k1 = t.cam_chunk_begin[v + 1];
    int k = k0 + rl;
    for (; k + 3 * kRowLanes < k1; k += 4 * kRowLanes) {
      float p[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) p[u] = partial[(long long)(k + u * kRowLanes) * C + c];
#pragma unroll
      for (int u = 0; u < 4; ++u) s += (double)p[u];
    }
    for (; k < k1; k += kRowLanes) s += (double)partial[(long long)k * C + c];
  }
  s_cam[cl][rl] = s;
  __syncthreads();
  double acc[3] = {0, 0, 0};
  if (rl == 0 && col_ok) {
    double tot = 0.0;
#pragma unroll
    for (int r = 0; r < kRowLanes; ++r) tot += s_cam[cl][r];
    const float mean = (float)(tot / (double)t.cam_tokens[v]);
    const double cur = (double)mean;
    const long long ip = (long long)(t.n_srows + v) * C + c;
    const double prev = (double)fp_prev[ip];
    acc[0] = cur * prev;
    acc[1] = cur * cur;
    acc[2] = prev * prev;
    fp_cur[ip] = mean;
  }
  block_reduce_n<3>(acc, s_red, -1);
  for (int g = 0; g < t.n_groups; ++g) {
    double* rec = records + ((long long)wg * kMaxGroups + g) * kRec;
    if (threadIdx.x == 0)
#pragma unroll
      for (int k = 0; k < kRec; ++k) rec[k] = (g == gv && k >= 5) ? acc[k >= 5 ? k - 5 : 0] : 0.0;
  }
}

__device__ __forceinline__ double cos_from(double dot, double nn, double pp) {
  double den = sqrt(nn) * sqrt(pp);
  return dot / fmax(den, 1e-12);
}

// One workgroup of 256 threads.  evaluate == 0: the block is computed without
// a test (warmup, forced pass, step-0 force, first visit): clear the flag and
// the staleness.
__global__ __launch_bounds__(256) void gate_decide_kernel(const double* __restrict__ records, int n_wg, GateArgs ga, GateState gs,
                                   int sb, int b, int evaluate) {
  const int lane = threadIdx.x;
  if (!evaluate) {
    if (lane == 0) {
      gs.flags[b] = 0;
      gs.stale[sb] = 0;
      if (gs.fp_sel != nullptr) gs.fp_sel[sb] ^= 1;  // computed: the current fingerprint becomes the cached one
    }
    return;
  }
  __shared__ double s_red[4 * kRec];
  double s_min = 1e300, d_max = -1e300;
  for (int g = 0; g < ga.n_groups; ++g) {
    // threads stride the workgroup records (one 64-byte record per load
    // batch, two batches in flight); fixed-shape reductions keep the sums
    // deterministic
    double tot[kRec] = {0, 0, 0, 0, 0, 0, 0, 0};
    auto add = [&](int w) __attribute__((always_inline)) {
      const double2* r2 = reinterpret_cast<const double2*>(records + ((long long)w * kMaxGroups + g) * kRec);
      double2 d[kRec / 2];
#pragma unroll
      for (int k = 0; k < kRec / 2; ++k) d[k] = r2[k];
#pragma unroll
      for (int k = 0; k < kRec / 2; ++k) {
        tot[2 * k] = (2 * k == 3) ? fmax(tot[2 * k], d[k].x) : tot[2 * k] + d[k].x;
        tot[2 * k + 1] = (2 * k + 1 == 3) ? fmax(tot[2 * k + 1], d[k].y) : tot[2 * k + 1] + d[k].y;
      }
    };
    int w = threadIdx.x;
    for (; w + 256 < n_wg; w += 512) {
      add(w);
      add(w + 256);
    }
    if (w < n_wg) add(w);
    block_reduce_n<kRec>(tot, s_red, 3);
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
  if (gs.fp_sel != nullptr && !skip) gs.fp_sel[sb] ^= 1;
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

int fp_compare_groups_of_wg(int C, int n_srows, int n_cams) {
  return (C + kFpCompareCols - 1) / kFpCompareCols * ((n_srows + kSpRows - 1) / kSpRows + n_cams);
}

void launch_fp_compare(const float* x, int C, const FpTables& t, const float* partial, float* fp0, float* fp1,
                       const int* sel, double* records, hipStream_t st) {
  dim3 grid((C + kFpCompareCols - 1) / kFpCompareCols, (t.n_srows + kSpRows - 1) / kSpRows + t.n_cams);
  fp_compare_kernel<<<grid, 256, 0, st>>>(x, C, t, partial, fp0, fp1, sel, records);
}

void launch_gate_decide(const double* records, int n_wg, const GateArgs& ga, const GateState& gs, int sb, int b,
                        int n_blocks, int evaluate, hipStream_t st) {
  (void)n_blocks;
  gate_decide_kernel<<<1, 256, 0, st>>>(records, n_wg, ga, gs, sb, b, evaluate);
}

}  // namespace xc
