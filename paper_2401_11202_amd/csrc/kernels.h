// Internal launch interface between the host planner (partir_api.cpp) and the
// HIP kernels.  Plain structs passed by value as kernel arguments.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace partir {

// Epilogue of a GEMM output tile.
enum GemmEpi : int {
  EPI_BF16 = 0,      // C (bf16) = act(acc + bias)
  EPI_F32 = 1,       // C (f32)  = act(acc + bias)
  EPI_PARTIAL = 2,   // partial[split] (f32) = acc        (split-K #sum)
  EPI_RESID_F32 = 3, // C (f32)  = resid + act(acc + bias) (resid may alias C)
  EPI_BF16_SAVE = 4  // C (bf16) = act(acc + bias) and aux (bf16) = acc + bias
};

// C = A . B^T over a grid of virtual shards.
//   A : [M, K] bf16 row-major, leading dim lda.
//   B : per group g, B_g^T stored [N, K] bf16 row-major (leading dim ldb).
//   C : per group g, [M, N] row-major (leading dim ldc).
// Shards: rm #tile shards along M (extent ms each), rn along N (extent ns),
// rk #sum shards along K (extent ks).  Output tiles never straddle a shard:
// tpm / tpn tiles per shard (the last one may be partial).
struct GemmParams {
  const uint16_t* A;
  const uint16_t* B[3];
  void* C[3];
  const float* bias[3];
  const float* resid;
  float* partial;
  void* aux;       // EPI_BF16_SAVE: pre-activation output (group 0, leading dim ldc)
  int64_t lda, ldb, ldc, ldr, part_ld, part_stride;
  int M, N, K, ngroups;
  int rm, ms, tpm;
  int rn, ns, tpn;
  int rk, ks;
  int tiles_m, tiles_n;
  int nsplit;      // 1: the rk shards accumulate in order in one accumulator
  int group_m;     // tile-order grouping for L2 reuse
  int act;         // 0 none, 1 gelu-erf
  int epi;         // GemmEpi
  // Load balance of the last, partial wave of output tiles (nsplit == 1):
  // tiles [tail_base, tiles_m * tiles_n) each run as tail_parts workgroups
  // over consecutive ranges of tail_kt 64-wide K tiles and store their fp32
  // accumulators to tail_ws ([tile - tail_base][part][128 x 512 floats]); the
  // fixup launch adds the parts in ascending order and runs the epilogue.
  // tail_parts <= 1: every tile in one workgroup.
  float* tail_ws;
  int tail_base, tail_parts, tail_kt;
  // Operand layouts: 0 K-contiguous (A [M, K], B^T [N, K]); 1 MN-major
  // (A stored [K, M] with leading dim lda, B stored [K, N] with leading dim
  // ldb).  MN-major operands take no activation.
  int a_mn, b_mn;
};

hipError_t launch_gemm_bf16(const GemmParams& p, hipStream_t s);
// The second launch of a GEMM with tail_parts > 1 (after launch_gemm_bf16 on
// the same stream).
hipError_t launch_gemm_bf16_fixup(const GemmParams& p, hipStream_t s);
// Bytes of tail_ws per tail part.
constexpr size_t kGemmTailPartBytes = 512 * 128 * 4;

// Operands held as separate device-local arrays (the lowered program's
// per-device arrays, Sec. 6): the GEMM reads and writes them in place, so an
// all_gather becomes addressing in the operand fetch and a reduce_scatter
// the owner's store.  A table with rows/cols 0 is unused (plain pointer).
//   a: A row blocks of a_rows rows (a_rows % 64 == 0), leading dim lda.
//   b: B^T blocks, b[g * b_gstride + nb * b_nk + kb] = group g's rows
//      [nb b_nrows, +b_nrows) and K columns [kb b_kcols, +b_kcols)
//      (b_nrows % 64 == 0, b_kcols % 64 == 0), each row-major with leading
//      dim ldb.
//   c: C row blocks of c_rows rows (c_rows % 16 == 0), leading dim ldc; with
//      EPI_RESID_F32 the residual is the part itself (C += result).
constexpr int kMaxParts = 64;
struct GemmParts {
  const uint16_t* a[kMaxParts];
  const uint16_t* b[kMaxParts];
  void* c[kMaxParts];
  int a_rows;
  int b_nrows, b_kcols, b_nk, b_gstride;
  int c_rows;
};
hipError_t launch_gemm_bf16_parts(const GemmParams& p, const GemmParts& t, hipStream_t s);
hipError_t launch_gemm_bf16_parts_fixup(const GemmParams& p, const GemmParts& t, hipStream_t s);
int gemm_bf16_tile_m();
int gemm_bf16_tile_n();

// fp32 GEMM: C = A . B with B [K, N] (b_nk = 0) or B^T [N, K] (b_nk = 1).
struct GemmF32Params {
  const float* A;
  const float* B;
  float* C;          // EPI_F32 output, or partial buffer base for EPI_PARTIAL
  int64_t lda, ldb, ldc, part_stride;
  int M, N, K;
  int b_nk;
  int rm, ms, tpm;
  int rn, ns, tpn;
  int rk, ks;
  int tiles_m, tiles_n;
  int nsplit;
  int epi;           // EPI_F32 or EPI_PARTIAL
};
hipError_t launch_gemm_f32(const GemmF32Params& p, hipStream_t s);
int gemm_f32_tile();

// Ordered split-K reduction: out = epilogue(sum_{r=0..R-1} partial[r]).
struct ReduceParams {
  const float* partial;
  int64_t part_ld, part_stride;
  int R, M, N;
  void* C;
  int64_t ldc;
  const float* bias;
  const float* resid;
  int64_t ldr;
  int act;
  int out_bf16;
  int resid_add;
};
hipError_t launch_splitk_reduce(const ReduceParams& p, hipStream_t s);

// Causal (or full) softmax attention, one head of d_head = 128 per block row.
//   Q, K, V, O: [B*S, ld] bf16 row-major; head h uses columns [h*128, h*128+128).
struct AttnParams {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  uint16_t* O;
  int64_t ldq, ldk, ldv, ldo;
  int B, S, H;       // sequences, length, heads (over all shards)
  int causal;
  float scale_log2;  // scale * log2(e)
  // key axis as a loop of nsplit shards (a custom associative #sum): shard s
  // covers key blocks [s * kb_per, (s + 1) * kb_per) of 64 keys and writes its
  // unnormalised output and softmax statistics instead of O.  With a causal
  // mask a shard is written only for the rows at or after its first key.
  int nsplit = 1;
  int kb_per = 0;
  float* Opart = nullptr;   // [nsplit][B*S][H*128] fp32, sum_j 2^(s_j c - m) v_j
  float* Mpart = nullptr;   // [nsplit][B*S][H] running max m (log2 domain, scaled)
  float* Lpart = nullptr;   // [nsplit][B*S][H] sum_j 2^(s_j c - m)
  // optional: the per-row base-2 log-sum-exp m + log2(l), [B*S][H] fp32,
  // kept for the backward pass (written by the unsplit kernel or the combine)
  float* lse = nullptr;
};
hipError_t launch_attention(const AttnParams& p, hipStream_t s);
// O = combine over the shards: M = max m_s, w_s = 2^(m_s - M),
// O = (sum_s w_s o_s) / (sum_s w_s l_s), s ascending; bf16 into p.O
hipError_t launch_attention_combine(const AttnParams& p, hipStream_t s);

// Gradients of the attention core (d_head = 128, S a multiple of 128) for
// the output cotangent dO, from the forward's O and its per-row base-2
// log-sum-exp lse[token][head] = log2 sum_j 2^(scale log2(e) s_j).  dQ, dK,
// dV bf16 in the layout of Q, K, V; Dstat [B*S][H] fp32 workspace (the
// rowsums of dO * O, written by the first pass, read by the second).
struct AttnBwdParams {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  const uint16_t* O;
  const uint16_t* dO;
  const float* lse;
  float* Dstat;
  uint16_t* dQ;
  uint16_t* dK;
  uint16_t* dV;
  int64_t ldq, ldk, ldv, ldo, ldg, lddq, lddk, lddv;
  int B, S, H;
  int causal;
  float scale;        // softmax scale
  float scale_log2;   // scale * log2(e)
};
hipError_t launch_attention_backward(const AttnBwdParams& p, hipStream_t s);

// y (bf16) = g * x / sqrt(mean(x^2) + eps), one row of D fp32 per wave.
struct RmsParams {
  const float* x;
  const float* g;
  uint16_t* y;
  int64_t ldx, ldy;
  int rows, D;
  float eps;
};
hipError_t launch_rmsnorm(const RmsParams& p, hipStream_t s);
// RMSNorm over rows held in device-local arrays: rows [i rows_part, (i+1)
// rows_part) of x are part x[i] (leading dim ldx); p.x is unused.
struct RmsParts {
  const float* x[kMaxParts];
  int rows_part;
};
hipError_t launch_rmsnorm_parts(const RmsParams& p, const RmsParts& t, hipStream_t s);


// Backward of H = act(Z) for Z, dH [rows, cols] bf16: dZ = dH * act'(Z)
// and H = act(Z), both [rows, cols] bf16 with leading dim ld (the weight
// gradients read them in place).  act 0 = identity, 1 = GELU-erf.  With
// colpart set, also the column sums of dZ (as stored, bf16) over each block
// of 64 rows: colpart[row block][col], the first stage of launch_colsum.
struct ActBwdParams {
  const uint16_t* Z;
  const uint16_t* dH;
  uint16_t* dZ;
  uint16_t* H;
  float* colpart;
  int64_t ld;
  int rows, cols;
  int act;
};
hipError_t launch_act_backward(const ActBwdParams& p, hipStream_t s);

// out[c] = sum over rows of in[r][c] (bf16 in, fp32 out), rows summed in
// blocks of 64 into partial[ceil(rows / 64)][cols], then the blocks in order:
// deterministic.  cols a multiple of 8.  partial_ready: the first stage was
// done by the producer of `in` (act_backward's colpart); only the second runs.
constexpr int kColSumChunk = 64;
struct ColSumParams {
  const uint16_t* in;
  float* partial;
  float* out;
  int64_t ld;
  int rows, cols;
  int partial_ready;
};
hipError_t launch_colsum(const ColSumParams& p, hipStream_t s);

}  // namespace partir
