// Internal declarations shared by the HIP kernels and the host orchestration.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace xc {

typedef __bf16 bf16;

// Maximum number of fingerprint view groups and conditioning values.
constexpr int kMaxGroups = 8;
constexpr int kMaxCond = 512;
constexpr int kMaxAction = 64;

// Columns per workgroup of the gate kernel.
constexpr int kFpCompareCols = 32;
// Doubles per (workgroup, group) partial record of the gate kernel.
constexpr int kFpRecord = 8;

// GEMM epilogue modes.
enum EpiMode : int {
  EPI_BIAS_F32 = 0,  // out_f32[m][n] = acc + bias[n]
  EPI_OPROJ = 1,     // out_f32 = resid + gate * (acc + bias)          (x1)
  EPI_UP = 2,        // out_t  = gelu_tanh(acc + bias)                   (u)
  EPI_DOWN = 3,      // out_f32 = resid + gate * (acc + bias)  (y); out_t = y - xin (cached residual)
  EPI_QKV = 4,       // acc + bias; per-head RMSNorm * gain on q and k; q -> q_out, k/v -> caches (bf16)
};

// 3-D rotary embedding tables (device).  Pair i of axis a (0 frame, 1 row,
// 2 column) at axis position p is tab[off[a] + p * np[a] + i] = (cos, sin) of
// the rotation angle.  The frame section is indexed by frame slot (one slot
// per (view group, frame) pair) and rebuilt for each generation; pos[row]
// packs the row's frame slot | h << 10 | w << 20.  tab == null: no rotation.
struct RopeArgs {
  const float2* tab;
  const int* pos;
  int np[3];
  int off[3];
};

// (cos, sin) of head pair `pair` for token `row`.
__device__ __forceinline__ float2 rope_cs(const RopeArgs& r, int row, int pair) {
  const int packed = r.pos[row];
  if (pair < r.np[0]) return r.tab[r.off[0] + (packed & 1023) * r.np[0] + pair];
  pair -= r.np[0];
  if (pair < r.np[1]) return r.tab[r.off[1] + ((packed >> 10) & 1023) * r.np[1] + pair];
  pair -= r.np[1];
  return r.tab[r.off[2] + ((packed >> 20) & 1023) * r.np[2] + pair];
}

struct EpiArgs {
  int M;               // valid rows
  int N;               // columns (row stride of every output)
  const float* bias;   // [N]
  float* out_f32;      // see EpiMode
  void* out_t;         // see EpiMode (element type = model dtype), may be null for EPI_DOWN
  const float* resid;  // [M][N]
  const float* gate;   // [N]
  const float* xin;    // [M][N]
  // EPI_QKV: column block j (C = H * D columns each) is part part_base + j
  // of (q, k, v): part_base 0 for the [q; k; v] projection, 1 for [k; v]
  int part_base;
  RopeArgs rope;       // rotation of q and k (tab == null: none)
  // EPI_DOWN, optional (null: off): per-camera column-sum partials of the
  // block output y and of the stored residual (the bf16 values), one pair of
  // rows per 32-row block of tokens: csum_part[kind][rb][slot][N], kind 0 = y,
  // 1 = residual, slot 0 = the camera of the block's first token, slot 1 = the
  // next camera, which starts at token offset rb_split[rb] (32: none)
  float* csum_part;
  const int* rb_split;
  int n_rb;
  const float* gq;     // [D]
  const float* gk;     // [D]
  void* q_out;         // [H][Mpad][D]
  void* k_cache;       // [H][Lcap][D], token m at row kv_off + m
  void* vt_cache;      // [H][D][Lcap], token m at column kv_off + m
  int H, D, Mpad, Lcap, kv_off;
};

// Global-channel sources of a gated evaluation (the column sums of the block
// input per camera), so that the comparison kernel need not read every token:
//   mode FULL: read x;
//   otherwise block b-1's skip flag selects: computed -> sum the 32-row-block
//   partials its MLP-down epilogue wrote (and, for a gateable b-1, refresh the
//   sums of its stored residual, csum_rhat[b-1]); skipped -> the input sums of
//   b-1 plus the sums of its stored residual (x_b = x_{b-1} + r_hat).
// Every evaluation leaves its input's sums in csum_in[b] for block b+1.
struct FoldArgs {
  int full;                  // 1: read x (no partials for this block)
  int b;
  int prev_gateable;
  const int* flags;          // [B] skip flags of this pass
  const float* csum_part;    // see EpiArgs
  int n_rb;
  const int* cam_rb_lo;      // [n_cams] first 32-row block holding a token of the camera
  const int* cam_rb_hi;      // [n_cams] one past the last such block
  const int* rb_cam;         // [n_rb] camera of each block's first token
  double* csum_in;           // [B][n_cams][C] this pass's input sums of each gated block (null: none kept)
  double* csum_rhat;         // [B][n_cams][C] residual sums of step t
};

// Per-pass gate hyper-parameters handed to the decision kernel.
struct GateArgs {
  int adaptive;
  float tau_floor, margin, alpha, tau_cos_fixed, tau_dev, eps;
  int max_stale;
  int strict0;          // 1 when this is step 0 in strict mode
  float tau_strict0;
  int n_groups;
  int action_dim;       // 0: no action channel this pass
  float action[kMaxAction];
  float action_prev[kMaxAction];
  int spatial_count[kMaxGroups];  // entries in each group's spatial fingerprint
};

// Gate state pointers (device).
struct GateState {
  float* ema;          // [S][B], NaN = unset
  int* stale;          // [S][B]
  int* skip_counts;    // [S][B]
  int* flags;          // [B] skip flag of the current pass
  int* rec_dec;        // [B] decision code of the last denoising pass
  float* rec_s;        // [B]
  float* rec_d;        // [B]
  float* rec_tau;      // [B]
  int* fp_sel;         // [S][B] refresh-on-compute mode: which fingerprint set holds (t, b)'s
                       // cached fingerprint, flipped when the block computes; null otherwise
};

// Fingerprint tables (device).
struct FpTables {
  int n_cams;
  const int* cam_row_begin;  // [n_cams + 1] first token row of each camera (prefix)
  int n_groups;
  const int* grp_srow_begin; // [G + 1] spatial fingerprint rows per group (prefix)
  const int* grp_cam_begin;  // [G + 1] cameras per group (prefix)
  int n_srows;
  const int* srows;          // [n_srows] global token row of each spatial row
};

// ---- launchers (each enqueues on `st`) -----------------------------------
void launch_cond(const float* action, int temb_dim, int action_dim, float timestep, float* cond_silu,
                 hipStream_t st);
void launch_adaln(int dtype, const void* w_ada, const float* b_ada, const float* cond_silu, int rows_per_block,
                  long long block_stride_w, int n_blocks, int dc, float* mod, hipStream_t st);
// rhat / skip_out: when the skip flag is set, write skip_out = x + rhat
// (the skip path) instead of returning at entry
void launch_ln_mod(int dtype, const float* x, const float* shift, const float* scale, void* out, int L, int C,
                   const int* flag, hipStream_t st, const void* rhat = nullptr, float* skip_out = nullptr);
void launch_gemm(int dtype, EpiMode mode, const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                 const int* flag, hipStream_t st);
// float32 models: per-head RMSNorm * gain of q and k (with the rotary
// embedding when rope.tab != null), q -> q [H][Mpad][D], k / v -> the caches
// at row / column kv_off + m.  qs, ks, vs: column 0 of each part in a
// row-major [L][ld] float32 matrix; a null part is skipped.
void launch_qk_norm(int dtype, const float* qs, const float* ks, const float* vs, int ld, const float* gq,
                    const float* gk, const RopeArgs& rope, void* q, void* kring, void* vtring, int L, int H, int D,
                    int Mpad, int Lcap, int kv_off, const int* flag, hipStream_t st);
// Rebuilds the rotary tables for generation n: frame slot s has position
// n * slot_frames[s] + slot_frame[s]; row and column sections hold positions
// 0 .. rows-1 and 0 .. cols-1, the three sections contiguous in that order
// (r.off = {0, n_slots * np[0], n_slots * np[0] + rows * np[1]}); theta: rotary
// base.
void launch_rope_table(float2* tab, const RopeArgs& r, int n_slots, const int* slot_frames, const int* slot_frame,
                       int rows, int cols, double theta, long long n, hipStream_t st);
// Floats of the attention workspace (partials of items whose keys are split
// across workgroups) for L queries over Lk keys, H heads of dimension D.
size_t attention_workspace_floats(int L, int Lk, int H, int D);
// ws: ws_floats floats of workspace; the key split is chosen among those
// whose partials fit (none: no split).
void launch_attention(int dtype, const void* q, const void* kring, const void* vtring, void* o, float* ws,
                      size_t ws_floats, int L, int Mpad, int Lcap, int Lk, int H, int D, const int* flag,
                      hipStream_t st);
void launch_axpby(float a, const float* x, float b, const float* y, float* out, long long n, hipStream_t st);
void launch_pass_begin(const GateState& gs, int n_blocks, hipStream_t st);
// Gated evaluation, first launch: fingerprint of x against the (t, b) cache
// and the refresh.  fp0 / fp1: the (t, b) fingerprint sets; with sel == null
// the cached fingerprint is fp0 and is overwritten in place, otherwise it is
// fp[*sel] and the current one goes to the other set.  records:
// gate_workgroups(...) * kMaxGroups * kFpRecord doubles.
int gate_workgroups(int C, int n_srows, int n_cams);
void launch_fp_compare(const float* x, int C, const FpTables& t, float* fp0, float* fp1, const int* sel,
                       double* records, const FoldArgs& fold, hipStream_t st);
// Second launch: the decision from the records of the first.
void launch_gate_decide(const double* records, int n_wg, const GateArgs& ga, const GateState& gs, int sb, int b,
                        int evaluate, hipStream_t st);
void launch_fill_f32(float* p, float v, long long n, hipStream_t st);
// out [H][R][D] float32 from a model-dtype cache [H][Lcap][D] (transposed = 0)
// or [H][D][Lcap] (transposed = 1), rows 0 .. R-1
void launch_read_cache(int dtype, const void* src, float* out, int H, int R, int D, long long Lcap, int transposed,
                       hipStream_t st);
// Register-only MFMA loop (shape 0: 32x32x16, 1: 16x16x32 bf16), timed with
// events on st; waits for it.
hipError_t mfma_rate(int shape, int random, hipStream_t st, double* tflops);
// global -> LDS stream of 24 KB stages with row_bytes (64 / 128 / 256) per
// row and request; allocates and frees a 33 MB source; waits for it.
hipError_t lds_dma_rate(int row_bytes, hipStream_t st, double* tbps);

}  // namespace xc
