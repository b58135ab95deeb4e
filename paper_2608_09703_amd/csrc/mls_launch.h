// Launch descriptors shared by the host planner (mls_api.cpp) and the kernel
// translation units. Plain structs passed by value as kernel arguments.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mls.h"

namespace mls {

constexpr int kMaxModels = 8;

// Tile of the fused logits kernels: BM vocabulary rows x BN token columns.
constexpr int kFusedBM = 128;      // general core
constexpr int kFusedWideBM = 128;  // wide bf16 core (all widths multiples of 64)
// forward partial records per (vocabulary tile, token, sub-model): one per
// wave row of the tile, each over its own half of the tile's rows
constexpr int kFusedFwdParts = 2;
// diagnostics records per (vocabulary tile, token), one per wave row likewise
constexpr int kDiagParts = 2;
constexpr int kFusedBN = 128;
// Tile of the backward GEMMs.
constexpr int kGemmBM = 128;
constexpr int kGemmBN = 128;

// Per-row partial statistics of one (sub-model, vocabulary tile, token):
//   x = max logit over the tile's vocabulary rows (own max)
//   y = sum exp(l - x)            (tau = 1)
//   z = sum exp((l - x) / tau)
//   w = sum e_v * l_v with e_v = exp((l_s,v - x_s) / tau) the teacher's
//       weights relative to the teacher's max x_s of the same tile
// (w of the teacher itself uses its own logits).
struct FusedArgs {
  int32_t M;
  int32_t teacher;
  int32_t order[kMaxModels];  // processing order; order[0] is the teacher
  const void* h[kMaxModels];
  const void* W[kMaxModels];
  int64_t d[kMaxModels];
  int64_t T;
  int64_t V;
  const int64_t* labels;
  int64_t ignore_index;
  float tau;
  float inv_tau;
  int32_t wide;  // 1: wide bf16 core (BM = kFusedWideBM)
  int32_t group_v;  // vocabulary tiles per ordering group (see tile_coords), >= 1
  int32_t n_tt;  // token tiles
  int32_t n_vt;  // vocabulary tiles in this launch
  // forward
  float4* partials;  // [M (processing order)][n_tt][n_vt * kFusedFwdParts][kFusedBN]
  // forward of the fused forward + backward: every logit, as fp16 of its
  // distance to its partial record's maximum, [M (sub-model index)][n_tt * BN][ld_lslab]
  uint16_t* lslab;
  int64_t ld_lslab;
  // backward
  const float* lse1;  // [M][T]
  const float* lset;  // [M][T]
  const int32_t* n_valid;
  const float* g_ce;  // device [M] or null
  const float* g_kl;
  float host_gce[kMaxModels];
  float host_gkl[kMaxModels];
  void* slab;   // [M][T_pad][Vc]  dJ/dlogits, token-major
  void* slabT;  // [M][Vc][T_pad]  dJ/dlogits, vocabulary-major
  int64_t T_pad;
  int64_t Vc;
  int64_t v0;  // first vocabulary row of the chunk
};

// One output matrix of a grouped NT GEMM: C[m][n] (+)= sum_k A[m][k] B[n][k].
// With Cb set the result goes to the bf16 matrix Cb instead, as
//   Cb[m][n] = bf16(sum + (Cpart ? Cpart[m][n] : 0) + (accumulate ? Cb[m][n] : 0))
// (Cpart: fp32 partial sums of earlier vocabulary chunks, same layout).
struct GemmGroup {
  const void* A;
  const void* B;
  float* C;
  uint16_t* Cb;
  const float* Cpart;
  int64_t lda;  // elements
  int64_t ldb;
  int64_t ldc;
  int64_t rows;  // m extent
  int64_t cols;  // n extent
  int64_t K;     // contraction length in elements (a multiple of the LDS row)
  int32_t tiles_m;
  int32_t tiles_n;
  int32_t tile_begin;
  int32_t accumulate;
  int32_t group_m;  // tile order: 0 = n fastest; g > 0 = groups of g row tiles, rows fastest
  // bf16 wide path only: operand layouts. 0: A is [m][k], B is [k][n] (grad_h:
  // slab [t][v] times a head chunk [v][d]); 1: A is [k][m], B is [k][n] (grad_W:
  // slab [t][v] as [k=t][m=v] times h [t][d]). rows/cols are the stored row counts
  // of A/B for these layouts (see WideMma::run).
  int32_t kind;
  int64_t ldc_rows;  // grad_W (kind 1): rows of C to write (the chunk's vocabulary rows)
};

constexpr int kMaxGemmGroups = 2 * kMaxModels;

struct GemmArgs {
  int32_t ngroups;
  // Tiles [0, phase_tiles) and [phase_tiles, total) have different costs (K);
  // each phase is spread evenly over the XCDs. 0 = one phase.
  int32_t phase_tiles;
  GemmGroup g[kMaxGemmGroups];
};

// dst[c][r] = src[(r0 + r) * ld_src + c] for r0 + r < src_rows, else 0;
// r < out_rows, c < cols; dst row stride ld_dst.
struct TransposeJob {
  const void* src;
  void* dst;
  int64_t ld_src;
  int64_t ld_dst;
  int64_t r0;
  int64_t src_rows;
  int64_t out_rows;
  int64_t cols;
};

struct TransposeArgs {
  int32_t njobs;
  TransposeJob j[kMaxModels];
};

struct RowArgs {
  int32_t M;
  int32_t teacher;
  const void* h[kMaxModels];
  const void* W[kMaxModels];
  int64_t d[kMaxModels];
  int64_t T;
  int64_t V;
  const int64_t* labels;
  int64_t ignore_index;
  float tau;
  int32_t order[kMaxModels];  // sub-model of each partial slot; order[0] is the teacher
  int32_t n_rec;           // partial records per token and sub-model
  // row merge: the forward chunk of tokens [t0, t0 + Tc) whose records follow
  int64_t t0;
  int64_t Tc;
  const float4* partials;  // [M slots][ceil(Tc / kFusedBN)][n_rec][kFusedBN]
  float* lab;              // [M][T] label logits
  float* stats;            // lse1, lset, ce_row, kl_row, h_row
  int32_t* header;         // n_valid, flags
  float* ce;
  float* kl;
  float* entropy;
};

// Logit gradient of one token chunk from its stored logits (fused forward +
// backward): the slab holds fp16 l - m (m: the partial record's maximum) and
// receives bf16 G in place.
struct GradArgs {
  int32_t M;
  int32_t order[kMaxModels];  // processing order of the records; order[0] is the teacher
  int64_t Tc;                 // tokens of the chunk (rows of the slab with data)
  int64_t Tc_pad;             // rows of each sub-model's slab
  int64_t t0;                 // first token of the chunk
  int64_t T;                  // all tokens (statistics row length)
  int64_t V;
  int64_t ld;                 // slab row length (>= V, a multiple of 8)
  const int64_t* labels;      // [T]
  int64_t ignore_index;
  float inv_tau;
  const float* lse1;          // [M][T]
  const float* lset;          // [M][T]
  const int32_t* n_valid;
  const float* g_ce;          // device [M] or null (host values then)
  const float* g_kl;
  float host_gce[kMaxModels];
  float host_gkl[kMaxModels];
  const float4* partials;     // [M slots][Tc_pad / kFusedBN][n_rec][kFusedBN]
  int32_t n_rec;
  uint16_t* slab;             // [M][Tc_pad][ld]
};

// Cross-model diagnostics (M <= kMaxDiagModels).
constexpr int kMaxDiagModels = 4;
constexpr int kDiagBN = 128;     // token tile, wide bf16 path
constexpr int kDiagGenBN = 64;   // token tile, general path
struct DiagArgs {
  int32_t M;
  const void* h[kMaxModels];
  const void* W[kMaxModels];
  int64_t d[kMaxModels];
  int64_t T;
  int64_t V;
  const int64_t* labels;
  int64_t ignore_index;
  int32_t n_tt;
  int32_t n_vt;
  int32_t group_v;        // tile order: vocabulary tiles per group
  float* partials;        // [n_vt * kDiagParts][M*M + 3M][T]
  float* rowvals;         // [T][2*M*M]
  float* kl_pair;         // [M][M]
  float* agree;           // [M][M]
  int32_t* argmax;        // [M][T] or null
};

// Scatter of one diagnostics pass over a subset of at most kMaxDiagModels
// sub-models (sub[k] is the sub-model of slot k) into the [M][M] outputs and
// the [M][T] argmax rows.
struct DiagScatterArgs {
  int32_t M;
  int32_t n;  // slots used
  int32_t sub[kMaxDiagModels];
  int64_t T;
  const float* kl_sub;     // [n][n]
  const float* agree_sub;  // [n][n]
  const int32_t* am_sub;   // [n][T] or null
  float* kl_pair;          // [M][M]
  float* agree;            // [M][M]
  int32_t* argmax;         // [M][T] or null
};

// Inter-model junction (eq. (1)).
struct JunctionArgs {
  int64_t T;
  int64_t d_prev;   // width of o
  int64_t d_fresh;  // width of e
  int32_t prev_first;
  int32_t accumulate;
  const void* o;    // [T][d_prev]
  const void* e;    // [T][d_fresh]
  void* x;          // [T][d_prev + d_fresh]
  const void* g_x;  // [T][d_prev + d_fresh]
  void* g_o;        // [T][d_prev]
  void* g_e;        // [T][d_fresh]
};

// Speculative-decoding head step.
struct HeadArgs {
  int64_t T;       // rows (tokens)
  int64_t V;
  int64_t d;
  const void* o;   // [T][d]
  const void* W;   // [V][d]
  float* logits;   // [T][V]
  int32_t n_tt;
  int32_t n_vt;
  int32_t group_v;
};
// Parameters of one row's sampling distribution.
struct RowDist {
  float m;      // max logit / temperature
  float total;  // sum of exp weights exp(l / temperature - m)
  float theta;  // nucleus threshold on the exp weight (0: keep every positive weight)
  int tie_cut;  // tokens with weight == theta are kept for index <= tie_cut
  float kept;   // sum of kept weights
};
struct SampleArgs {
  int64_t rows;
  int64_t V;
  float inv_temp;
  float top_p;
  int32_t greedy;
  const float* logits;  // [rows][V]
  const float* u;       // [rows]
  int32_t* tokens;      // [rows]
  RowDist* params;      // [rows] distribution records, or nullptr
};
struct RowParamArgs {
  int64_t rows0;          // rows of logits0, then rows1 rows of logits1
  int64_t rows1;
  int64_t V;
  float inv_temp;
  float top_p;
  const float* logits0;
  const float* logits1;
  RowDist* params;        // [rows0 + rows1]
};
struct VerifyArgs {
  const RowDist* dparams;  // draft rows [gamma][batch]
  const RowDist* tparams;  // verifier rows [batch][gamma + 1]
  int64_t batch;
  int64_t V;
  int32_t gamma;
  int32_t greedy;
  float inv_temp;
  float top_p;
  const float* draft_logits;   // [gamma][batch][V] (one row per draft step and sequence)
  const float* target_logits;  // [batch][gamma + 1][V]
  const int32_t* draft_tokens; // [gamma][batch]
  const float* u_accept;       // [gamma][batch]
  const float* u_sample;       // [batch]
  int32_t* n_accepted;         // [batch]
  int32_t* next_token;         // [batch]
};

// MFMA ceiling probe (measurement aid).
hipError_t launch_mfma_probe(int random, int iters, float* sink, hipStream_t stream);
double mfma_probe_flops(int iters);
int64_t mfma_probe_sink_floats();

// Sets the calling thread's mls_last_error text to "what: detail" and returns s.
mls_status set_error(mls_status s, const char* what, const char* detail);

// Launchers (each enqueues on `stream` and returns the launch status).
int fused_tile_rows(bool wide);
hipError_t launch_fused_fwd(const FusedArgs& a, bool f32, hipStream_t stream);
hipError_t launch_fused_bwd(const FusedArgs& a, bool f32, hipStream_t stream);
// Output tile of the backward GEMMs (wide bf16 path or the general path).
int gemm_tile_rows(bool wide);
int gemm_tile_cols(bool wide);
// Wide bf16 path: grad_h and grad_W products read in stored layouts.
hipError_t launch_gemm_wide(const GemmArgs& a, int total_tiles, hipStream_t stream);
hipError_t launch_gemm_nt(const GemmArgs& a, int total_tiles, bool f32, hipStream_t stream);
hipError_t launch_transpose(const TransposeArgs& a, int64_t max_out_rows, int64_t max_cols,
                            bool f32, hipStream_t stream);
int gemm_wide_k_tile();  // K values per K-tile of the wide gradient GEMM
int diag_tile_rows(bool wide);
int diag_tile_cols(bool wide, int M);
int diag_record_floats(int M);
hipError_t launch_diag_tiles(const DiagArgs& a, bool f32, bool wide, hipStream_t stream);
hipError_t launch_diag_reduce(const DiagArgs& a, hipStream_t stream);
hipError_t launch_diag_scatter(const DiagScatterArgs& a, hipStream_t stream);
bool junction_shape(int64_t width, int* tpr, int* cpl);
int64_t junction_max_width();
hipError_t launch_junction_fwd(const JunctionArgs& a, bool act_f32, hipStream_t stream);
hipError_t launch_junction_bwd(const JunctionArgs& a, bool act_f32, bool grad_f32, hipStream_t stream);
int head_tile();  // token rows of a head tile
int head_tile_rows(bool wide, int n_tt);  // vocabulary rows of a head tile (128 or 192)
int row_elems_per_thread(int64_t V);
// rows: head_tile_rows(wide, a.n_tt) on the wide bf16 path, else 128 (checked)
hipError_t launch_head_logits(const HeadArgs& a, bool f32, bool wide, int rows,
                              hipStream_t stream);
hipError_t launch_sample(const SampleArgs& a, int ept, hipStream_t stream);
hipError_t launch_row_params(const RowParamArgs& a, int ept, hipStream_t stream);
hipError_t launch_verify(const VerifyArgs& a, int ept, hipStream_t stream);
hipError_t launch_label_logits(const RowArgs& a, bool f32, hipStream_t stream);
hipError_t launch_finalize_rows(const RowArgs& a, hipStream_t stream);
hipError_t launch_reduce_losses(const RowArgs& a, hipStream_t stream);
hipError_t launch_count_valid(const RowArgs& a, hipStream_t stream);
hipError_t launch_grad_logits(const GradArgs& a, hipStream_t stream);

}  // namespace mls
