// HBM-bound kernels of the block: conditioning, adaLN modulation GEMV,
// LayerNorm + modulation, QK RMSNorm with the scatter into the KV cache,
// the cached-residual add of a skipped block and the sampler axpby.
//
// Every kernel that belongs to a block's compute path takes `flag`: when it is
// non-null and the block's skip flag is set, the kernel returns at entry
// (wave-uniformly), so a skipped block costs one empty launch.
#include "xc_internal.h"

#include <math.h>

namespace xc {

namespace {

// Sum over the 64 lanes of a wave without LDS round trips: lane pairs and quads by DPP quad
// permutations, quad pairs and 8-lane halves by the DPP row mirrors, then the
// row pairs and the two half-waves by the permlane swaps.  Every step adds
// two values that the partner lane adds in the other order, so every lane
// ends with the same total, in the same order in every run.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_move<0xB1>(v);    // quad_perm [1,0,3,2]: lane ^ 1
  v += dpp_move<0x4E>(v);    // quad_perm [2,3,0,1]: lane ^ 2
  v += dpp_move<0x141>(v);   // row_half_mirror: quad 0 <-> quad 1 of each 8 lanes
  v += dpp_move<0x140>(v);   // row_mirror: the two 8-lane halves of each row
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

template <typename T>
__device__ __forceinline__ T to_t(float v);
template <>
__device__ __forceinline__ float to_t<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16 to_t<bf16>(float v) { return (bf16)v; }

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(bf16 v) { return (float)v; }

// c = [temb(timestep); action]; cond_silu = SiLU(c).  temb is the sinusoidal
// embedding [cos(tau f_i), sin(tau f_i)], f_i = 10000^(-i/h), h = temb_dim/2,
// evaluated in double so the large arguments (tau up to 1000) keep full
// float accuracy.
struct CondArgs {
  float action[kMaxAction];
};

__global__ void cond_kernel(CondArgs a, int temb_dim, int action_dim, float timestep, float* cond_silu) {
  const int h = temb_dim / 2;
  for (int j = threadIdx.x; j < temb_dim + action_dim; j += blockDim.x) {
    double c;
    if (j < h) {
      c = cos((double)timestep * exp(-log(10000.0) * (double)j / (double)h));
    } else if (j < temb_dim) {
      c = sin((double)timestep * exp(-log(10000.0) * (double)(j - h) / (double)h));
    } else {
      c = (double)a.action[j - temb_dim];
    }
    cond_silu[j] = (float)(c / (1.0 + exp(-c)));
  }
}

// mod[blk][r] = sum_j W_ada[blk][r][j] * cond_silu[j] + b_ada[blk][r].  A wave
// takes 8 consecutive output rows and issues all their 16-byte weight loads
// before any arithmetic (lane l reads elements [V l, V l + V) of each row, V =
// 16 / sizeof(T); when V does not divide the row length the rows go
// element-wise), then reduces the 8 dot products across the wave.
template <typename T>
__global__ __launch_bounds__(256) void adaln_kernel(const T* __restrict__ w, const float* __restrict__ b,
                                                    const float* __restrict__ cond_silu, int rows_per_block,
                                                    long long block_stride_w, long long block_stride_b,
                                                    int n_rows_total, int dc, float* __restrict__ mod) {
  constexpr int V = 16 / sizeof(T);
  constexpr int kRowsPerWave = 8;
  typedef T tvec __attribute__((ext_vector_type(V)));
  __shared__ float s_c[kMaxCond];
  for (int j = threadIdx.x; j < dc; j += blockDim.x) s_c[j] = cond_silu[j];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int row0 = (blockIdx.x * 4 + wave) * kRowsPerWave;
  // whole 16-byte chunks per row (rows start 16-byte aligned only when V divides dc)
  const int n_chunks = dc % V == 0 ? dc / V : 0;
  float acc[kRowsPerWave];
#pragma unroll
  for (int rr = 0; rr < kRowsPerWave; ++rr) acc[rr] = 0.f;
  for (int j0 = 0; j0 < n_chunks; j0 += 64) {
    const int j = j0 + lane;
    tvec v[kRowsPerWave];
#pragma unroll
    for (int rr = 0; rr < kRowsPerWave; ++rr) {
      const int row = row0 + rr;
      if (row < n_rows_total && j < n_chunks) {
        const int blk = row / rows_per_block, r = row - blk * rows_per_block;
        v[rr] = *reinterpret_cast<const tvec*>(w + blk * block_stride_w + (long long)r * dc + (long long)j * V);
      } else {
#pragma unroll
        for (int e = 0; e < V; ++e) v[rr][e] = (T)0.f;
      }
    }
    if (j < n_chunks)
#pragma unroll
      for (int rr = 0; rr < kRowsPerWave; ++rr)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[rr] += to_f(v[rr][e]) * s_c[j * V + e];
  }
  for (int jt = n_chunks * V + lane; jt < dc; jt += 64)
#pragma unroll
    for (int rr = 0; rr < kRowsPerWave; ++rr) {
      const int row = row0 + rr;
      if (row < n_rows_total) {
        const int blk = row / rows_per_block, r = row - blk * rows_per_block;
        acc[rr] += to_f(w[blk * block_stride_w + (long long)r * dc + jt]) * s_c[jt];
      }
    }
#pragma unroll
  for (int rr = 0; rr < kRowsPerWave; ++rr) acc[rr] = wave_sum(acc[rr]);
  if (lane < kRowsPerWave) {
    float a = acc[0];
#pragma unroll
    for (int rr = 1; rr < kRowsPerWave; ++rr) a = lane == rr ? acc[rr] : a;
    const int row = row0 + lane;
    if (row < n_rows_total) {
      const int blk = row / rows_per_block, r = row - blk * rows_per_block;
      mod[row] = a + b[blk * block_stride_b + r];
    }
  }
}

// The same GEMV when a row of W_ada is a whole number of 16-byte chunks (every
// supported conditioning width): the weights of all blocks form one
// contiguous [rows][dc] matrix, and a wave takes 32 consecutive rows, i.e.
// one contiguous span of 32 * cpr chunks, walked lane-linearly (every load
// instruction reads 1 KB of consecutive bytes).  Each chunk's dot product with
// its slice of SiLU(c) goes to LDS; lane r < 32 then sums row r's cpr
// partials in order (deterministic).
template <typename T>
__global__ __launch_bounds__(256) void adaln_flat_kernel(const T* __restrict__ w, const float* __restrict__ b,
                                                         const float* __restrict__ cond_silu, int n_rows, int dc,
                                                         float* __restrict__ mod) {
  constexpr int V = 16 / sizeof(T);
  constexpr int kRows = 32;   // rows per wave
  constexpr int kBatch = 8;   // chunk loads in flight per lane
  typedef T tvec __attribute__((ext_vector_type(V)));
  __shared__ float s_c[kMaxCond];
  extern __shared__ float s_part[];  // [4 waves][kRows * cpr]
  for (int j = threadIdx.x; j < dc; j += blockDim.x) s_c[j] = cond_silu[j];
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int cpr = dc / V;  // chunks per row
  const long long row0 = ((long long)blockIdx.x * 4 + wave) * kRows;
  if (row0 >= n_rows) return;
  const int rows = (int)min((long long)kRows, n_rows - row0);
  const int n_chunks = rows * cpr;
  const tvec* src = reinterpret_cast<const tvec*>(w + row0 * dc);
  float* part = s_part + wave * kRows * cpr;
  for (int c0 = 0; c0 < n_chunks; c0 += 64 * kBatch) {
    tvec v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int c = c0 + u * 64 + lane;
      if (c < n_chunks) v[u] = src[c];
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int c = c0 + u * 64 + lane;
      if (c < n_chunks) {
        const int k = c % cpr;
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < V; ++e) acc += to_f(v[u][e]) * s_c[k * V + e];
        part[c] = acc;
      }
    }
  }
  // lanes read partials other lanes of this wave wrote: LDS operations of one
  // wave complete in order, the fence keeps the compiler from reordering them
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
  if (lane < rows) {
    float a = 0.f;
    for (int k = 0; k < cpr; ++k) a += part[lane * cpr + k];
    mod[row0 + lane] = a + b[row0 + lane];
  }
}

// h = LayerNorm(x) * (1 + scale) + shift per row (no affine, biased variance,
// eps 1e-6), one wave per row, values held in registers between the passes.
// With a skip flag that is set the block is skipped: the kernel then writes
// the skip path's output skip_out = x + rhat (Eq. 4) for its rows instead
// when skip_out is given (the first LayerNorm of a gated block evaluation),
// else returns at entry.  skip_out may alias x (element-wise, in place).
template <typename T, int MAXV>
__global__ __launch_bounds__(256) void ln_mod_kernel(const float* x, const float* __restrict__ shift,
                                                     const float* __restrict__ scale, T* __restrict__ out, int L,
                                                     int C, const int* __restrict__ flag,
                                                     const T* __restrict__ rhat, float* skip_out) {
  const bool skip = flag != nullptr && *flag;
  if (skip && skip_out == nullptr) return;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= L) return;
  const int C4 = C >> 2;
  const float4* xr = reinterpret_cast<const float4*>(x + (long long)row * C);
  if (skip) {
    typedef T T4 __attribute__((ext_vector_type(4)));
    const T4* rr = reinterpret_cast<const T4*>(rhat + (long long)row * C);
    float4* orow = reinterpret_cast<float4*>(skip_out + (long long)row * C);
#pragma unroll
    for (int i = 0; i < MAXV; ++i) {
      const int c4 = lane + i * 64;
      if (c4 < C4) {
        const float4 a = xr[c4];
        const T4 r = rr[c4];
        orow[c4] = make_float4(a.x + to_f(r[0]), a.y + to_f(r[1]), a.z + to_f(r[2]), a.w + to_f(r[3]));
      }
    }
    return;
  }
  float4 v[MAXV];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    int c4 = lane + i * 64;
    if (c4 < C4) {
      v[i] = xr[c4];
      s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
    }
  }
  const float mu = wave_sum(s) / (float)C;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    int c4 = lane + i * 64;
    if (c4 < C4) {
      float a = v[i].x - mu, bb = v[i].y - mu, c = v[i].z - mu, d = v[i].w - mu;
      q += (a * a + bb * bb) + (c * c + d * d);
    }
  }
  const float var = wave_sum(q) / (float)C;
  const float rstd = 1.0f / sqrtf(var + 1e-6f);
  // four consecutive outputs per lane leave as one 8-byte (bf16) or 16-byte store
  typedef T T4 __attribute__((ext_vector_type(4)));
  T4* orow = reinterpret_cast<T4*>(out + (long long)row * C);
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    int c4 = lane + i * 64;
    if (c4 < C4) {
      float4 sc = reinterpret_cast<const float4*>(scale)[c4];
      float4 sh = reinterpret_cast<const float4*>(shift)[c4];
      T4 o;
      o[0] = to_t<T>((v[i].x - mu) * rstd * (1.f + sc.x) + sh.x);
      o[1] = to_t<T>((v[i].y - mu) * rstd * (1.f + sc.y) + sh.y);
      o[2] = to_t<T>((v[i].z - mu) * rstd * (1.f + sc.z) + sh.z);
      o[3] = to_t<T>((v[i].w - mu) * rstd * (1.f + sc.w) + sh.w);
      orow[c4] = o;
    }
  }
}

// QK RMSNorm and scatter.  Input: qkv [Mpad][3C] float (bias added).  One
// workgroup per (64-token tile, head):
//   q  -> rms(q) * gq       -> Q  [H][Mpad][D]
//   k  -> rms(k) * gk       -> K  cache [H][Lcap][D] at row kv_off + m
//   v                       -> V^T cache [H][D][Lcap] at column kv_off + m
// The V tile is transposed through LDS so the V^T rows are written coalesced.
template <typename T>
__global__ __launch_bounds__(256) void qk_norm_kernel(const float* __restrict__ qs, const float* __restrict__ ks,
                                                      const float* __restrict__ vs, int ld,
                                                      const float* __restrict__ gq, const float* __restrict__ gk,
                                                      RopeArgs rope, T* __restrict__ q, T* __restrict__ kring,
                                                      T* __restrict__ vtring, int L, int H, int D, int Mpad,
                                                      int Lcap, int kv_off, const int* __restrict__ flag) {
  if (flag != nullptr && *flag) return;
  __shared__ float s_v[64][129];
  const int tile = blockIdx.x, h = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m0 = tile * 64;
  // q and k: each wave takes 16 tokens; lane holds head dims lane, lane + 64
  for (int i = 0; i < 16; ++i) {
    int tl = wave * 16 + i;
    int m = m0 + tl;
    if (m >= L) break;
#pragma unroll
    for (int part = 0; part < 2; ++part) {
      const float* base = part == 0 ? qs : ks;
      if (base == nullptr) continue;
      const float* src = base + (long long)m * ld + h * D;
      const float* g = part == 0 ? gq : gk;
      float a0 = lane < D ? src[lane] : 0.f;
      float a1 = lane + 64 < D ? src[lane + 64] : 0.f;
      float ss = wave_sum(a0 * a0 + a1 * a1);
      float r = 1.0f / sqrtf(ss / (float)D + 1e-6f);
      a0 = lane < D ? a0 * r * g[lane] : 0.f;
      a1 = lane + 64 < D ? a1 * r * g[lane + 64] : 0.f;
      if (rope.tab != nullptr) {
        // pair (2j, 2j+1) sits in lanes (2j, 2j+1): (a, b) -> (a c - b s, a s + b c)
        const float p0 = __shfl_xor(a0, 1, 64), p1 = __shfl_xor(a1, 1, 64);
        const float sgn = (lane & 1) ? 1.f : -1.f;
        if (lane < D) {
          const float2 cs = rope_cs(rope, m, lane >> 1);
          a0 = a0 * cs.x + sgn * p0 * cs.y;
        }
        if (lane + 64 < D) {
          const float2 cs = rope_cs(rope, m, (lane + 64) >> 1);
          a1 = a1 * cs.x + sgn * p1 * cs.y;
        }
      }
      T* dst = part == 0 ? q + ((long long)h * Mpad + m) * D : kring + ((long long)h * Lcap + kv_off + m) * D;
      if (lane < D) dst[lane] = to_t<T>(a0);
      if (lane + 64 < D) dst[lane + 64] = to_t<T>(a1);
    }
    if (vs != nullptr) {
      const float* vsrc = vs + (long long)m * ld + h * D;
      if (lane < D) s_v[tl][lane] = vsrc[lane];
      if (lane + 64 < D) s_v[tl][lane + 64] = vsrc[lane + 64];
    }
  }
  if (vs == nullptr) return;
  __syncthreads();
  // V^T: row dd holds 64 consecutive tokens
  const int nt = min(64, L - m0);
  for (int idx = threadIdx.x; idx < D * 64; idx += 256) {
    int dd = idx >> 6, tl = idx & 63;
    if (tl < nt) vtring[((long long)h * D + dd) * Lcap + kv_off + m0 + tl] = to_t<T>(s_v[tl][dd]);
  }
}

// Rotary tables (see RopeArgs): entry idx of the contiguous frame / row /
// column sections gets (cos, sin) of position * theta^(-2i/d_a), evaluated in
// double (frame positions grow with the generation index).
__global__ void rope_table_kernel(float2* __restrict__ tab, RopeArgs r, int n_slots,
                                  const int* __restrict__ slot_frames, const int* __restrict__ slot_frame, int rows,
                                  int cols, double log_theta, long long n) {
  const int n0 = n_slots * r.np[0], n1 = rows * r.np[1], n2 = cols * r.np[2];
  for (int idx = blockIdx.x * blockDim.x + threadIdx.x; idx < n0 + n1 + n2; idx += gridDim.x * blockDim.x) {
    double pos;
    int i, np;
    if (idx < n0) {
      const int s = idx / r.np[0];
      i = idx - s * r.np[0];
      np = r.np[0];
      pos = (double)n * slot_frames[s] + slot_frame[s];
    } else if (idx < n0 + n1) {
      const int k = idx - n0, p = k / r.np[1];
      i = k - p * r.np[1];
      np = r.np[1];
      pos = p;
    } else {
      const int k = idx - n0 - n1, p = k / r.np[2];
      i = k - p * r.np[2];
      np = r.np[2];
      pos = p;
    }
    const double ang = pos * exp(-2.0 * i / (2.0 * np) * log_theta);
    tab[idx] = make_float2((float)cos(ang), (float)sin(ang));
  }
}

__global__ void axpby_kernel(float a, const float* __restrict__ x, float b, const float* __restrict__ y,
                             float* __restrict__ out, long long n) {
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < n; i += (long long)gridDim.x * 256)
    out[i] = a * x[i] + b * y[i];
}

// out[h][r][d] (float32, r < R) from a cache stored [H][Lcap][D] or, when
// transposed, [H][D][Lcap] (row r is column r)
template <typename T>
__global__ void read_cache_kernel(const T* __restrict__ src, float* __restrict__ out, int R, int D, long long Lcap,
                                  int transposed, long long n) {
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < n; i += (long long)gridDim.x * 256) {
    const long long hr = i / D, h = hr / R;
    const int d = (int)(i - hr * D), r = (int)(hr - h * R);
    const long long j = transposed ? ((h * D + d) * Lcap + r) : ((h * Lcap + r) * D + d);
    out[i] = (float)src[j];
  }
}

__global__ void fill_f32_kernel(float* p, float v, long long n) {
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < n; i += (long long)gridDim.x * 256) p[i] = v;
}

__global__ void pass_begin_kernel(GateState gs, int n_blocks) {
  for (int b = threadIdx.x; b < n_blocks; b += blockDim.x) {
    gs.rec_dec[b] = 2;  // forced unless a decision kernel evaluates the block
    gs.rec_s[b] = __builtin_nanf("");
    gs.rec_d[b] = __builtin_nanf("");
    gs.rec_tau[b] = __builtin_nanf("");
    gs.flags[b] = 0;
  }
}

int grid_for(long long n, int per_block) {
  long long g = (n + per_block - 1) / per_block;
  if (g > 8192) g = 8192;
  if (g < 1) g = 1;
  return (int)g;
}

}  // namespace

void launch_cond(const float* action, int temb_dim, int action_dim, float timestep, float* cond_silu,
                 hipStream_t st) {
  CondArgs a;
  for (int i = 0; i < kMaxAction; ++i) a.action[i] = i < action_dim ? action[i] : 0.f;
  cond_kernel<<<1, 256, 0, st>>>(a, temb_dim, action_dim, timestep, cond_silu);
}

void launch_adaln(int dtype, const void* w_ada, const float* b_ada, const float* cond_silu, int rows_per_block,
                  long long block_stride_w, int n_blocks, int dc, float* mod, hipStream_t st) {
  // W_ada is [n_blocks][rows_per_block][dc] and b_ada [n_blocks][rows_per_block]:
  // block_stride_w = rows_per_block * dc, the bias stride is rows_per_block.
  int total = rows_per_block * n_blocks;
  const int esz = dtype == 1 ? 2 : 4;
  if ((dc * esz) % 16 == 0 && block_stride_w == (long long)rows_per_block * dc) {
    const int grid = (total + 127) / 128;  // 4 waves x 32 rows
    const size_t lds = (size_t)4 * 32 * (dc * esz / 16) * sizeof(float);
    if (dtype == 1)
      adaln_flat_kernel<bf16><<<grid, 256, lds, st>>>((const bf16*)w_ada, b_ada, cond_silu, total, dc, mod);
    else
      adaln_flat_kernel<float><<<grid, 256, lds, st>>>((const float*)w_ada, b_ada, cond_silu, total, dc, mod);
    return;
  }
  int grid = (total + 31) / 32;  // 4 waves x 8 rows
  if (dtype == 1)
    adaln_kernel<bf16><<<grid, 256, 0, st>>>((const bf16*)w_ada, b_ada, cond_silu, rows_per_block, block_stride_w,
                                             rows_per_block, total, dc, mod);
  else
    adaln_kernel<float><<<grid, 256, 0, st>>>((const float*)w_ada, b_ada, cond_silu, rows_per_block,
                                              block_stride_w, rows_per_block, total, dc, mod);
}

void launch_ln_mod(int dtype, const float* x, const float* shift, const float* scale, void* out, int L, int C,
                   const int* flag, hipStream_t st, const void* rhat, float* skip_out) {
  int grid = (L + 3) / 4;
  int maxv = (C / 4 + 63) / 64;
#define XC_LN(T, MV) \
  ln_mod_kernel<T, MV><<<grid, 256, 0, st>>>(x, shift, scale, (T*)out, L, C, flag, (const T*)rhat, skip_out)
  if (dtype == 1) {
    if (maxv <= 2) XC_LN(bf16, 2);
    else if (maxv <= 8) XC_LN(bf16, 8);
    else XC_LN(bf16, 16);
  } else {
    if (maxv <= 2) XC_LN(float, 2);
    else if (maxv <= 8) XC_LN(float, 8);
    else XC_LN(float, 16);
  }
#undef XC_LN
}

void launch_qk_norm(int dtype, const float* qs, const float* ks, const float* vs, int ld, const float* gq,
                    const float* gk, const RopeArgs& rope, void* q, void* kring, void* vtring, int L, int H, int D,
                    int Mpad, int Lcap, int kv_off, const int* flag, hipStream_t st) {
  dim3 grid((L + 63) / 64, H);
  if (dtype == 1)
    qk_norm_kernel<bf16><<<grid, 256, 0, st>>>(qs, ks, vs, ld, gq, gk, rope, (bf16*)q, (bf16*)kring,
                                               (bf16*)vtring, L, H, D, Mpad, Lcap, kv_off, flag);
  else
    qk_norm_kernel<float><<<grid, 256, 0, st>>>(qs, ks, vs, ld, gq, gk, rope, (float*)q, (float*)kring,
                                                (float*)vtring, L, H, D, Mpad, Lcap, kv_off, flag);
}

void launch_rope_table(float2* tab, const RopeArgs& r, int n_slots, const int* slot_frames, const int* slot_frame,
                       int rows, int cols, double theta, long long n, hipStream_t st) {
  const int total = n_slots * r.np[0] + rows * r.np[1] + cols * r.np[2];
  rope_table_kernel<<<(total + 255) / 256, 256, 0, st>>>(tab, r, n_slots, slot_frames, slot_frame, rows, cols,
                                                         log(theta), n);
}

void launch_axpby(float a, const float* x, float b, const float* y, float* out, long long n, hipStream_t st) {
  axpby_kernel<<<grid_for(n, 256 * 4), 256, 0, st>>>(a, x, b, y, out, n);
}

void launch_read_cache(int dtype, const void* src, float* out, int H, int R, int D, long long Lcap, int transposed,
                       hipStream_t st) {
  const long long n = (long long)H * R * D;
  if (dtype == 1)
    read_cache_kernel<bf16><<<grid_for(n, 256 * 4), 256, 0, st>>>((const bf16*)src, out, R, D, Lcap, transposed, n);
  else
    read_cache_kernel<float><<<grid_for(n, 256 * 4), 256, 0, st>>>((const float*)src, out, R, D, Lcap, transposed, n);
}

void launch_fill_f32(float* p, float v, long long n, hipStream_t st) {
  fill_f32_kernel<<<grid_for(n, 256 * 4), 256, 0, st>>>(p, v, n);
}

void launch_pass_begin(const GateState& gs, int n_blocks, hipStream_t st) {
  pass_begin_kernel<<<1, 256, 0, st>>>(gs, n_blocks);
}

}  // namespace xc
