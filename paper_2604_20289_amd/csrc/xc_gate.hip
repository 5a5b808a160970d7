// Fingerprint reduction and the dual-metric gate (Section 2.3-2.5), two
// launches per gated block evaluation.
//
// fp_compare : a 1-D grid of (32-column slice) x (spatial row chunks +
//              cameras) workgroups.
//   * spatial workgroups gather 16 fingerprint rows of the block input x for
//     their 32 columns, compare them with the cached fingerprint and write
//     the current rows over the refreshed set;
//   * camera workgroups read every token row of one camera for their 32
//     columns (the HBM-bound part: one read of x in total), form the token
//     mean (global channel) and compare it likewise;
//   * each workgroup leaves one partial record per view group (Eq. 5-6 terms:
//     dot, norms, max |delta|, sum |prev|).
// gate_decide: one workgroup; reduces all records in a fixed order
//   (deterministic), forms s = min-cosine and d = max-deviation, applies the
//   adaptive threshold (Eq. 8-9), the skip rule (Eq. 7) and the staleness
//   bound, and writes the block's skip flag, its staleness counter and the
//   statistics.  (A last-workgroup ticket inside fp_compare would save the
//   launch, but every workgroup would then need a device-scope release,
//   which on this chip writes back its XCD's L2: far slower than a launch.)
//
// Fingerprint storage for one (t, b): [n_srows + n_cams][C] float -- the
// spatial rows in group order, then one token-mean row per camera.
#include "xc_internal.h"

#include <math.h>

namespace xc {

namespace {

constexpr int kRec = kFpRecord;  // dot_s, nn_s, pp_s, maxabs_s, sumabs_prev_s, dot_g, nn_g, pp_g

// Block reduction of NF fields at once (NW waves): the per-field shuffle
// chains are independent, so their latencies overlap; one LDS exchange
// across the waves.  Field `max_field` takes the maximum, the
// others the sum; fixed order throughout.
template <int NF, int NW = 4>
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
    for (int w = 1; w < NW; ++w) r = f == max_field ? fmax(r, s_red[w * NF + f]) : r + s_red[w * NF + f];
    v[f] = r;
  }
}

__device__ __forceinline__ double cos_from(double dot, double nn, double pp) {
  double den = sqrt(nn) * sqrt(pp);
  return dot / fmax(den, 1e-12);
}

constexpr int kCmpThreads = 512;                      // threads of a comparison workgroup
constexpr int kCmpWaves = kCmpThreads / 64;
constexpr int kSpRows = 2 * (kCmpThreads / kFpCompareCols);  // spatial rows per workgroup
constexpr int kColGroups = kFpCompareCols / 4;       // float4 column groups of a camera workgroup
constexpr int kCamLanes = kCmpThreads / kColGroups;   // row lanes of a camera workgroup
constexpr int kCamUnroll = 8;                         // row loads in flight per lane

// The decision (last workgroup).  evaluate == 0: the block is computed
// without a test (warmup, forced pass, step-0 force, first visit): clear the
// flag and the staleness.
__device__ void decide(const double* records, int n_wg, const GateArgs& ga, const GateState& gs, int sb, int b,
                       int evaluate, double* s_red) {
  const int lane = threadIdx.x;
  if (!evaluate) {
    if (lane == 0) {
      gs.flags[b] = 0;
      gs.stale[sb] = 0;
      if (gs.fp_sel != nullptr) gs.fp_sel[sb] ^= 1;  // computed: the current fingerprint becomes the cached one
    }
    return;
  }
  // the per-(t, b) state the tail needs, fetched now so its latency overlaps
  // the record reduction (the records were written on every XCD: each load
  // round trip goes past this XCD's L2)
  float ema0 = 0.f;
  int stale0 = 0;
  if (lane == 0) {
    ema0 = gs.ema[sb];
    stale0 = gs.stale[sb];
  }
  double s_min = 1e300, d_max = -1e300;
  for (int g = 0; g < ga.n_groups; ++g) {
    // threads stride the workgroup records (64 bytes each), up to kBatch
    // records per thread loaded in one round; fixed-shape reductions keep
    // the sums deterministic
    constexpr int kBatch = 4;
    double tot[kRec] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int w0 = 0; w0 < n_wg; w0 += 256 * kBatch) {
      double2 d[kBatch][kRec / 2];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int w = w0 + u * 256 + (int)threadIdx.x;
        const double2* r2 = reinterpret_cast<const double2*>(records + ((long long)min(w, n_wg - 1) * kMaxGroups + g) * kRec);
#pragma unroll
        for (int k = 0; k < kRec / 2; ++k) d[u][k] = r2[k];
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (w0 + u * 256 + (int)threadIdx.x >= n_wg) continue;
#pragma unroll
        for (int k = 0; k < kRec / 2; ++k) {
          tot[2 * k] = (2 * k == 3) ? fmax(tot[2 * k], d[u][k].x) : tot[2 * k] + d[u][k].x;
          tot[2 * k + 1] = (2 * k + 1 == 3) ? fmax(tot[2 * k + 1], d[u][k].y) : tot[2 * k + 1] + d[u][k].y;
        }
      }
    }
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
  double ema = (double)ema0;
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
  const int stale = stale0;
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

// 512 threads; workgroup w takes column slice w % n_cs and row part
// w / n_cs: part y < n_sp handles spatial fingerprint rows [32 y, 32 y + 32)
// (two per lane), part n_sp + v the token mean of camera v (64 row lanes x 8
// float4 column lanes, every lane summing every 64th row with up to 8 loads
// in flight; lane sums combined in lane order through LDS).  (Measured at
// the multi-camera shape: 512 threads beat 256 and 1024.)  Every workgroup writes one record per group (zeros for
// the terms it does not own).
__global__ __launch_bounds__(kCmpThreads) void fp_compare_kernel(const float* __restrict__ x, int C, FpTables t, float* fp0,
                                                         float* fp1, const int* sel, double* __restrict__ records,
                                                         FoldArgs fold) {
  // cached fingerprint and where the current one goes
  const bool flip = sel != nullptr && *sel != 0;
  const float* fp_prev = flip ? fp1 : fp0;
  float* fp_cur = sel == nullptr ? fp0 : (flip ? fp0 : fp1);
  __shared__ double s_red[kCmpWaves * kRec];
  __shared__ double s_cam[kFpCompareCols][kCamLanes + 1];
  const int n_cs = (C + kFpCompareCols - 1) / kFpCompareCols;
  const int slice = blockIdx.x % n_cs, part = blockIdx.x / n_cs;
  const int wg = blockIdx.x;
  const int n_sp = (t.n_srows + kSpRows - 1) / kSpRows;
  if (part < n_sp) {
    const int cl = threadIdx.x % kFpCompareCols;
    const int rl = threadIdx.x / kFpCompareCols;
    constexpr int kRowLanes = kCmpThreads / kFpCompareCols;
    const int c = slice * kFpCompareCols + cl;
    const bool col_ok = c < C;
    const int i0 = part * kSpRows;
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
      block_reduce_n<5, kCmpWaves>(acc, s_red, 3);
      if (threadIdx.x == 0)
#pragma unroll
        for (int k = 0; k < kRec; ++k) rec[k] = k < 5 ? acc[k < 5 ? k : 0] : 0.0;
    }
  } else {
    const int v = part - n_sp;
    int gv = 0;
    while (gv + 1 < t.n_groups && t.grp_cam_begin[gv + 1] <= v) ++gv;
    const int r0 = t.cam_row_begin[v], r1 = t.cam_row_begin[v + 1];
    // this camera's column sums, lane l of the slice's first kFpCompareCols
    // threads holding column slice * kFpCompareCols + l (fixed-order sums)
    double tot = 0.0;
    if (fold.full) {
      const int cg = threadIdx.x % kColGroups, rl = threadIdx.x / kColGroups;
      const int c0 = slice * kFpCompareCols + cg * 4;
      double sx = 0.0, sy = 0.0, sz = 0.0, sw = 0.0;
      if (c0 < C) {
        const float* col = x + c0;
        for (int r = r0 + rl; r < r1; r += kCamUnroll * kCamLanes) {
          float4 p[kCamUnroll];
#pragma unroll
          for (int u = 0; u < kCamUnroll; ++u) {
            const int rr = r + u * kCamLanes;
            p[u] = rr < r1 ? *reinterpret_cast<const float4*>(col + (long long)rr * C) : make_float4(0.f, 0.f, 0.f, 0.f);
          }
#pragma unroll
          for (int u = 0; u < kCamUnroll; ++u) {
            sx += (double)p[u].x;
            sy += (double)p[u].y;
            sz += (double)p[u].z;
            sw += (double)p[u].w;
          }
        }
      }
      s_cam[cg * 4 + 0][rl] = sx;
      s_cam[cg * 4 + 1][rl] = sy;
      s_cam[cg * 4 + 2][rl] = sz;
      s_cam[cg * 4 + 3][rl] = sw;
      __syncthreads();
      if (threadIdx.x < kFpCompareCols)
        for (int l = 0; l < kCamLanes; ++l) tot += s_cam[threadIdx.x][l];
    } else {
      // from block b-1: the partials of its output (computed) or its input
      // sums plus its stored residual's sums (skipped)
      const int cl = threadIdx.x % kFpCompareCols, kl = threadIdx.x / kFpCompareCols;
      constexpr int kLanes = kCmpThreads / kFpCompareCols;
      const int c = slice * kFpCompareCols + cl;
      const long long cv = ((long long)(fold.b - 1) * t.n_cams + v) * C + c;
      if (fold.flags[fold.b - 1] == 0) {
        const int lo = fold.cam_rb_lo[v], hi = fold.cam_rb_hi[v];
        const long long kind = (long long)fold.n_rb * 2 * C;
        double sy = 0.0, sd = 0.0;
        if (c < C)
          for (int rb = lo + kl; rb < hi; rb += kLanes) {
            const long long o = ((long long)rb * 2 + (fold.rb_cam[rb] == v ? 0 : 1)) * C + c;
            sy += (double)fold.csum_part[o];
            sd += (double)fold.csum_part[kind + o];
          }
        s_cam[cl][kl] = sy;
        s_cam[cl][kLanes + kl] = sd;
        __syncthreads();
        if (threadIdx.x < kFpCompareCols && c < C) {
          double td = 0.0;
          for (int l = 0; l < kLanes; ++l) {
            tot += s_cam[threadIdx.x][l];
            td += s_cam[threadIdx.x][kLanes + l];
          }
          if (fold.prev_gateable) fold.csum_rhat[cv] = td;
        }
      } else if (threadIdx.x < kFpCompareCols && c < C) {
        tot = fold.csum_in[cv] + fold.csum_rhat[cv];
      }
    }
    double acc[3] = {0, 0, 0};
    const int c = slice * kFpCompareCols + threadIdx.x;
    if (threadIdx.x < kFpCompareCols && c < C) {
      if (fold.csum_in != nullptr) fold.csum_in[((long long)fold.b * t.n_cams + v) * C + c] = tot;
      const float mean = (float)(tot / (double)(r1 - r0));
      const double cur = (double)mean;
      const long long ip = (long long)(t.n_srows + v) * C + c;
      const double prev = (double)fp_prev[ip];
      acc[0] = cur * prev;
      acc[1] = cur * cur;
      acc[2] = prev * prev;
      fp_cur[ip] = mean;
    }
    block_reduce_n<3, kCmpWaves>(acc, s_red, -1);
    for (int g = 0; g < t.n_groups; ++g) {
      double* rec = records + ((long long)wg * kMaxGroups + g) * kRec;
      if (threadIdx.x == 0)
#pragma unroll
        for (int k = 0; k < kRec; ++k) rec[k] = (g == gv && k >= 5) ? acc[k >= 5 ? k - 5 : 0] : 0.0;
    }
  }
}

// One workgroup of 256 threads: the decision from all partial records.
__global__ __launch_bounds__(256) void gate_decide_kernel(const double* __restrict__ records, int n_wg, GateArgs ga,
                                                          GateState gs, int sb, int b, int evaluate) {
  __shared__ double s_red[4 * kRec];
  decide(records, n_wg, ga, gs, sb, b, evaluate, s_red);
}

}  // namespace

int gate_workgroups(int C, int n_srows, int n_cams) {
  return (C + kFpCompareCols - 1) / kFpCompareCols * ((n_srows + kSpRows - 1) / kSpRows + n_cams);
}

void launch_fp_compare(const float* x, int C, const FpTables& t, float* fp0, float* fp1, const int* sel,
                       double* records, const FoldArgs& fold, hipStream_t st) {
  const int grid = gate_workgroups(C, t.n_srows, t.n_cams);
  fp_compare_kernel<<<grid, kCmpThreads, 0, st>>>(x, C, t, fp0, fp1, sel, records, fold);
}

void launch_gate_decide(const double* records, int n_wg, const GateArgs& ga, const GateState& gs, int sb, int b,
                        int evaluate, hipStream_t st) {
  gate_decide_kernel<<<1, 256, 0, st>>>(records, n_wg, ga, gs, sb, b, evaluate);
}

}  // namespace xc
