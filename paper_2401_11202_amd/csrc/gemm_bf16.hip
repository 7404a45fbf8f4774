// bf16 MFMA GEMM for gfx950: C = A . B^T, A K-contiguous or stored [K, M],
// B K-contiguous or stored [K, N].
//
// One workgroup computes a 256x256 output tile of one virtual shard with eight
// waves (2 x 4, two per SIMD), each owning a 128x64 sub-tile as 8 x 4
// accumulators of v_mfma_f32_16x16x32_bf16.  K advances in 64-wide tiles
// through LDS buffers filled by buffer loads that write LDS directly (no
// register staging).  With A K-contiguous (every forward product) the two
// waves of a SIMD take turns: one runs a K tile's MFMAs on fragments already
// in its registers while the other reads its next fragments and issues the
// loads (the main loop below).  With A stored [K, M] (weight gradients) all
// eight waves run in step through two 64 KiB stages.  Out-of-range lanes
// (ragged M / N / K edges, tiles past the end) read as zeros.  The 256x256
// tile is the largest whose fp32 accumulators fit the register file, which
// keeps L2 -> LDS traffic per FLOP minimal.
//
// Loop semantics realised here (PartIR:Core, Sec. 5 / App. C):
//  * #tile over M or N: the grid enumerates every shard's tiles; a tile never
//    straddles a shard and stores into the shard's slice of C.
//  * #sum over K, fused: the shards' K-ranges are consecutive, so one tile's
//    K loop walks shard 0, 1, ..., R-1 in order into one accumulator.
//  * #sum over K, split: the grid also enumerates the K shards and each writes
//    its own fp32 partial; an ordered reduction (elementwise.hip) sums them.
#include "kernels.h"
#include "device_math.h"
#include "lds_dma.h"

// s_waitcnt with only the LDS / scalar-memory counter constrained (gfx9 encoding)
#define WAIT_LGKMCNT(n) __builtin_amdgcn_s_waitcnt((((n) & 15) << 8) | 0xF | (0x3 << 14) | (0x7 << 4))

namespace partir {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 256, BN = 256, NT = 512;
constexpr int BK = 64, NS = 2;
constexpr int PP_LDS = 160 * 1024;   // LDS of the two-group main loop
// Epilogue staging of the output tile in LDS (reusing the K stages): bf16
// rows of 256 + 8 elements (528 B, 16-byte aligned rows), fp32 in two halves
// of 128 rows of 256 + 4 floats (1040 B); the pads spread consecutive rows
// over the LDS banks.
constexpr int CPB = BN + 8, CPF = BN + 4;
constexpr int C_LDS = (BM * CPB * 2 > (BM / 2) * CPF * 4) ? BM * CPB * 2 : (BM / 2) * CPF * 4;
constexpr uint32_t OOB = 0x80000000u;          // offset that reads as zero
// GELU for bf16 outputs: Phi(x) by linear interpolation in an LDS table of
// (Phi(x_i), Phi(x_i+1) - Phi(x_i)), x_i = -6 + i/256, i < 3072, whose entries
// come from gelu_erf's erfc approximation.  Interpolation error <= h^2/8 max
// |Phi''| = 4.6e-7 (h = 1/256), so |GELU error| <= 5.4e-7 |x|, far below the
// bf16 rounding of the stored value; outside [-6, 6) Phi is 0 or 1 to
// 1e-9.  Nine VALU operations and one LDS read instead of one reciprocal,
// one exponential and twelve VALU operations.
constexpr int PHI_N = 3072;
constexpr float PHI_LO = -6.0f, PHI_SCALE = 256.0f;
constexpr int PHI_BYTES = PHI_N * 8;

template <typename T>
__device__ __forceinline__ T pick3(int g, T a, T b, T c) { return g == 0 ? a : (g == 1 ? b : c); }

// LDS tile layout: [row][64 k] = 128-byte rows of eight 16-byte chunks; chunk
// c of row r sits at position c ^ swz(r), swz(r) = bit1(r) | bit3(r) << 1 |
// bit2(r) << 2.  A fragment read takes 16 rows (lane % 16) at 4 chunks
// (lane / 16); the LDS serves it 8 lanes of each half-wave at a time, i.e.
// 8 rows at two chunks 2 apart, and swz gives the 4 rows of each parity
// distinct bits 0 and 2, so the 16 reads hit 16 different bank groups (as do
// any 16 consecutive lanes: the 8 rows of each parity get all 8 values).
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 1) | (((r >> 3) & 1) << 1) | (((r >> 2) & 1) << 2); }
// MN-major tile layout: [k][256 columns] = 512-byte rows of 32 chunks; chunk
// c of k row r sits at position c ^ mn_swz(r).  A transposed fragment read
// covers 4 k rows x 16 columns per 16-lane group, groups 0 and 1 (one pass)
// on rows 8 apart: the 4 (r & 3) term spreads the 4 rows over the banks, the
// 2 bit3(r) term keeps the two groups apart.
__device__ __forceinline__ int mn_swz(int r) { return (4 * (r & 3)) ^ (2 * ((r >> 3) & 1)); }

// PARTS: operands in device-local arrays (`t`, a kernel argument); else the
// plain pointers of `p` and t is unused.
// FIX: the fixup launch of a tail-split GEMM (no K loop: the accumulators are
// the sum of the stored parts).  AMN / BMN: A stored [K, M] / B stored [K, N]
// (row-major, the tile's 256 columns contiguous) instead of K-contiguous.
template <int EPI, int ACT, int PARTS, int FIX, int AMN = 0, int BMN = 0>
__device__ __forceinline__ void gemm_body(const GemmParams& p, const GemmParts* tb) {
  static_assert(!(PARTS && (AMN || BMN)), "device-local arrays are K-contiguous");
  constexpr int OPB = BM * BK * 2, STAGE = 2 * OPB, KK = BK / 32, RB = 1024 / (BK * 2) /* rows per 1 KiB */;
  constexpr int CPR = BK / 8;   // 16-byte chunks per row
  constexpr int MAIN = (NS * STAGE > C_LDS) ? NS * STAGE : C_LDS;
  constexpr bool PHI_TAB = ACT && (EPI == EPI_BF16 || EPI == EPI_BF16_SAVE);
  // PP: the two-group main loop below (every K-contiguous A); it uses all
  // 160 KiB of LDS for its buffers and builds the Phi table after the loop,
  // behind the epilogue's staging area
  constexpr bool PP = !FIX && !AMN;
  static_assert(C_LDS + PHI_BYTES <= PP_LDS, "epilogue staging and Phi table fit the PP buffers");
  constexpr int PHI_OFF = PP ? C_LDS : MAIN;
  constexpr int LDS_BYTES = PP ? PP_LDS : MAIN + (PHI_TAB ? PHI_BYTES : 0);
  __shared__ __attribute__((aligned(1024))) char smem[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: LDS bases and M0 in SGPRs
  const int wm = wave >> 2, wn = wave & 3;

  // ---- which tile of which virtual shard ----------------------------------
  const int ntiles = p.tiles_m * p.tiles_n;
  int bid = blockIdx.x;
  const int nwg = gridDim.x;
  int tail_unit = -1, tail_part = 0;   // K part of a tail tile
  if (FIX) {
    bid = p.tail_base + blockIdx.x;
  } else if (p.tail_parts > 1) {
    // XCD x (workgroups go round-robin to the 8 XCDs, in launch order) takes
    // a contiguous run of the whole tiles, then a contiguous run of the tail
    // parts, so every XCD gets the same share of both and the parts run last
    const int nf = p.tail_base, nu = nwg - nf;
    if (((nf | nu) & 7) == 0) {
      const int x = bid & 7, i = bid >> 3;
      bid = (i < (nf >> 3)) ? x * (nf >> 3) + i : nf + x * (nu >> 3) + (i - (nf >> 3));
    }
    if (bid >= nf) {
      tail_unit = bid - nf;
      tail_part = tail_unit % p.tail_parts;
      bid = nf + tail_unit / p.tail_parts;
    }
  } else if ((nwg & 7) == 0) {
    // Give each XCD a contiguous run of the tile order so neighbouring tiles
    // share that XCD's L2.
    bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  }
  const int split = bid / ntiles;
  const int tix = bid - split * ntiles;
  const int per_group = p.group_m * p.tiles_n;
  const int gidx = tix / per_group;
  const int first_m = gidx * p.group_m;
  const int gm = min(p.tiles_m - first_m, p.group_m);
  const int rr = tix - gidx * per_group;
  const int tm = first_m + rr % gm;
  const int tn = rr / gm;

  const int sm = tm / p.tpm, tmi = tm - sm * p.tpm;
  const int row0 = sm * p.ms + tmi * BM;
  const int rows = min(BM, p.ms - tmi * BM);
  const int per_gn = p.rn * p.tpn;
  const int grp = tn / per_gn, rem = tn - grp * per_gn;
  const int sn = rem / p.tpn, tni = rem - sn * p.tpn;
  const int col0 = sn * p.ns + tni * BN;
  const int cols = min(BN, p.ns - tni * BN);
  int k_begin = (p.nsplit > 1) ? split * p.ks : 0;
  int k_end = (p.nsplit > 1) ? k_begin + p.ks : p.K;
  if (tail_unit >= 0) {
    k_begin = tail_part * p.tail_kt * BK;
    k_end = min(p.K, k_begin + p.tail_kt * BK);
  }

  // Phi table (read after the main loop's barriers)
  auto build_phi = [&] {
    float2* tab = (float2*)(smem + PHI_OFF);
    for (int i = threadIdx.x; i < PHI_N; i += NT) {
      const float x0 = PHI_LO + (float)i / PHI_SCALE, x1 = PHI_LO + (float)(i + 1) / PHI_SCALE;
      const float p0 = phi_cdf(x0), p1 = phi_cdf(x1);
      tab[i] = make_float2(p0, p1 - p0);
    }
  };
  if (PHI_TAB && !PP) build_phi();

  // ---- global -> LDS loads ----------------------------------------------------
  // Per k tile each wave issues 4 + 4 wave-wide 16-byte loads; load j of wave
  // w fills rows 64 j + 8 w .. +8 of the operand tile (1 KiB of LDS written
  // lane by lane).  Lane L takes row +L/8, LDS chunk L%8, i.e. global chunk
  // (L%8) ^ swz(row).  One descriptor per 64-row block bounds the valid rows.
  const uint16_t* Bg = pick3(grp, p.B[0], p.B[1], p.B[2]);
  const uint16_t* At = p.A + (int64_t)row0 * p.lda;
  const uint16_t* Btile = Bg + (int64_t)col0 * p.ldb;
  constexpr int NJ = BM / (8 * RB);   // wave loads per operand per k tile
  constexpr int BLK = 8 * RB;          // rows covered by one load of all 8 waves
  static_assert(BLK == 64, "part tables assume 64-row load blocks");
  const GemmParts* const t = tb;
  __amdgpu_buffer_rsrc_t ra[NJ], rb[NJ];
  // start of the B row block j in K part kp (parts: the owning array; a block
  // with no valid rows takes any part's address, its descriptor reads nothing)
  auto b_block = [&](int j, int kp) -> const uint16_t* {
    if (PARTS && t->b_nrows) {
      const int gb = grp * t->b_gstride;
      if (cols - BLK * j <= 0) return t->b[gb + kp];
      const int n = col0 + BLK * j;
      const int nb = n / t->b_nrows;
      return t->b[gb + nb * t->b_nk + kp] + (int64_t)(n - nb * t->b_nrows) * p.ldb;
    }
    return Btile + (int64_t)BLK * j * p.ldb;
  };
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int va = min(max(rows - BLK * j, 0), BLK), vb = min(max(cols - BLK * j, 0), BLK);
    const uint16_t* a_blk = At + (int64_t)BLK * j * p.lda;
    if (PARTS && t->a_rows) {
      const int r = row0 + BLK * min(j, (rows - 1) / BLK);   // blocks past the rows: size 0 below
      const int ab = r / t->a_rows;
      a_blk = t->a[ab] + (int64_t)(r - ab * t->a_rows) * p.lda;
    }
    ra[j] = make_rsrc(a_blk, (uint32_t)(va * p.lda * 2));
    rb[j] = make_rsrc(b_block(j, 0), (uint32_t)(vb * p.ldb * 2));
  }
  // K part the B descriptors point into and where it ends (loads are issued
  // in increasing K, so the part only ever advances)
  int b_kpart = 0;
  int b_kend = (PARTS && t->b_nrows) ? t->b_kcols : 0;
  const int lrow = RB * wave + lane / CPR;
  const int lchunk = (lane % CPR) ^ swz(lrow);
  const uint32_t a_voff = (uint32_t)(lrow * p.lda * 2 + lchunk * 16);
  const uint32_t b_voff = (uint32_t)(lrow * p.ldb * 2 + lchunk * 16);
  const int lds_w = wave * 1024;
  const int nk = (k_end - k_begin + BK - 1) / BK;
  // MN-major operands: the LDS tile holds 64 k rows of 512 B (the 256 tile
  // columns).  Load j of wave w fills k rows 16 j + 2 w and +1 (the same
  // 1 KiB of LDS as in the K-contiguous layout); lane L takes row +L/32 and
  // LDS chunk L%32 = global chunk (L%32) ^ 4 (row & 3), which makes the
  // transposed fragment reads below conflict-free.  A descriptor per k tile
  // bounds the rows at the end of K (rows past it read as zero).
  const int mn_r = 2 * wave + (lane >> 5);
  const int mn_chunk = (lane & 31) ^ mn_swz(mn_r);
  const uint32_t a_mvoff = AMN ? (uint32_t)(mn_r * p.lda * 2 + mn_chunk * 16) : 0u;
  const uint32_t b_mvoff = BMN ? (uint32_t)(mn_r * p.ldb * 2 + mn_chunk * 16) : 0u;
  auto gload = [&](int kt, int stage) {
    const int kb = k_begin + kt * BK;
    if constexpr (AMN || BMN) {
      const uint32_t kvalid = (uint32_t)min(max(k_end - kb, 0), BK);
      char* base = smem + stage * STAGE + lds_w;
      __amdgpu_buffer_rsrc_t rma, rmb;
      if (AMN) rma = make_rsrc(p.A + (int64_t)kb * p.lda + row0, kvalid * (uint32_t)p.lda * 2);
      if (BMN) rmb = make_rsrc(Bg + (int64_t)kb * p.ldb + col0, kvalid * (uint32_t)p.ldb * 2);
      const uint32_t kmask = (kb + lchunk * 8 < k_end) ? 0u : OOB;
      const uint32_t so = (uint32_t)kb * 2;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        if (AMN)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rma, (lds_void*)(base + j * 8192), 16,
                                                   a_mvoff + (uint32_t)(j * 32 * p.lda), 0, 0, 0);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(ra[j], (lds_void*)(base + j * 8192), 16, a_voff | kmask, so, 0, 0);
        if (BMN)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rmb, (lds_void*)(base + OPB + j * 8192), 16,
                                                   b_mvoff + (uint32_t)(j * 32 * p.ldb), 0, 0, 0);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rb[j], (lds_void*)(base + OPB + j * 8192), 16, b_voff | kmask, so,
                                                   0, 0);
      }
      return;
    }
    const uint32_t kmask = (kb + lchunk * 8 < k_end) ? 0u : OOB;   // ragged K tail / past the end
    const uint32_t so = (uint32_t)kb * 2;   // A (and unparted B): K offset in bytes
    uint32_t so_b = so;
    if (PARTS && t->b_nrows) {
      // the all_gather of B along K: K tiles never straddle a part (a tail
      // part may start several parts in)
      if (kb >= b_kend && b_kpart + 1 < t->b_nk) {
        while (kb >= b_kend && b_kpart + 1 < t->b_nk) {
          ++b_kpart;
          b_kend += t->b_kcols;
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int vb = min(max(cols - BLK * j, 0), BLK);
          rb[j] = make_rsrc(b_block(j, b_kpart), (uint32_t)(vb * p.ldb * 2));
        }
      }
      so_b = (uint32_t)(kb - (b_kend - t->b_kcols)) * 2;
    }
    char* base = smem + stage * STAGE + lds_w;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra[j], (lds_void*)(base + j * 8192), 16, a_voff | kmask, so, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb[j], (lds_void*)(base + OPB + j * 8192), 16, b_voff | kmask, so_b, 0, 0);
    }
  };

  // ---- MFMA operand reads -----------------------------------------------------
  // v_mfma_f32_16x16x32_bf16 with the B fragment as the first operand: a
  // fragment is 16 rows (of A or B^T) x 32 k, lane l holding row l % 16 at
  // k = 8 (l / 16) .. +7, and the 16 x 16 result leaves lane l with output row
  // l % 16 at the 4 consecutive output columns 4 (l / 16) .. +3.
  const int fsw = swz(lane & 15);
  const int g16 = lane >> 4;
  const int a_rd = (wm * 128 + (lane & 15)) * BK * 2;
  const int b_rd = OPB + (wn * 64 + (lane & 15)) * BK * 2;

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.0f;

  // MN-major fragment of 16 columns from bc, k step ks (32 k rows): group G
  // = l / 16 reads k rows 32 ks + 8 G + (j16 >> 2) (and +4 for the high
  // half), columns bc + 4 (j16 & 3) .. +3; ds_read_b64_tr_b16 hands lane j16
  // of the group one column over the group's 4 rows, i.e. lane l holds
  // column bc + l % 16 at k = 32 ks + 8 (l / 16) + 0..7, the layout of a
  // K-contiguous fragment.
  const int j16 = lane & 15;
  const int mn_row = 8 * g16 + (j16 >> 2);
  const int mn_sw = mn_swz(mn_row);
  const int mn_col = 4 * (j16 & 3);
  auto mn_frag = [&](const char* op, int ks, int bc) -> bf16x8 {
    const int col = bc + mn_col;
    const char* pl = op + (32 * ks + mn_row) * 512 + (((col >> 3) ^ mn_sw) << 4) + ((col & 4) << 1);
    const i16x4 lo = lds_read_tr16(pl);
    const i16x4 hi = lds_read_tr16(pl + 4 * 512);
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  // fragments of one 32-wide k step: 8 A row blocks and 4 B row blocks
  bf16x8 fa0[8], fb0[4], fa1[8], fb1[4];
  auto ldfrag = [&](int stage, int ks, bf16x8* a, bf16x8* b) {
    const char* st = smem + stage * STAGE;
    const int ko = ((4 * ks + g16) ^ fsw) << 4;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      a[i] = AMN ? mn_frag(st, ks, wm * 128 + i * 16) : *(const bf16x8*)(st + a_rd + i * 16 * BK * 2 + ko);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      b[j] = BMN ? mn_frag(st + OPB, ks, wn * 64 + j * 16) : *(const bf16x8*)(st + b_rd + j * 16 * BK * 2 + ko);
  };
  // LDS reads per k step (a transposed fragment takes two)
  constexpr int NRD = (AMN ? 16 : 8) + (BMN ? 8 : 4);
  // B as the first operand: each lane ends up holding 4 consecutive output
  // columns of one output row.
  auto mma = [&](const bf16x8* a, const bf16x8* b) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
  };
  // instruction interleaving hints: mask bits MFMA 0x8, VMEM read 0x20, DS read 0x100
#define SGB(mask, n) __builtin_amdgcn_sched_group_barrier(mask, n, 0)
  // one k step: each of the 32 MFMAs followed by one of the next step's LDS
  // reads and, when refilling, one of the global loads
#define SLOTS(rf)                                              \
  _Pragma("unroll") for (int sl = 0; sl < 32; ++sl) {          \
    SGB(0x8, 1);                                               \
    if (sl < NRD) SGB(0x100, 1);                               \
    if ((rf) && sl < LPS) SGB(0x20, 1);                        \
  }

  constexpr int LPS = 2 * NJ;   // wave loads per k tile
  // prologue: both stages in flight, then wait for tile 0.  In the loop, the
  // first KK-1 steps of a tile read the next step's fragments while their
  // MFMAs run; then (tile kt+1 landed, every wave done with this stage) the
  // stage is refilled with tile kt+2 and the next tile's first fragments are
  // read during the last step.
  if constexpr (!FIX && !PP) {
#pragma unroll
  for (int s = 0; s < NS; ++s) gload(s, s);
  WAIT_VMCNT(LPS * (NS - 1));
  __syncthreads();
  ldfrag(0, 0, fa0, fb0);
  // One k tile; `refill` issues the loads of tile kt+NS (skipped once that
  // tile lies past the end, so no LDS write is still in flight at exit).
  auto tile = [&](int kt, int stage, bool refill) {
    const int next = (stage + 1 == NS) ? 0 : stage + 1;
#pragma unroll
    for (int kk = 0; kk < KK - 1; ++kk) {
      if (kk & 1) { ldfrag(stage, kk + 1, fa0, fb0); mma(fa1, fb1); }
      else { ldfrag(stage, kk + 1, fa1, fb1); mma(fa0, fb0); }
      SLOTS(false);
    }
    WAIT_VMCNT(LPS * (NS - 2));
    __syncthreads();
    if (refill) gload(kt + NS, stage);
    if ((KK - 1) & 1) { ldfrag(next, 0, fa0, fb0); mma(fa1, fb1); }
    else { ldfrag(next, 0, fa1, fb1); mma(fa0, fb0); }
    SLOTS(refill);
    return next;
  };
  int stage = 0, kt = 0;
  for (; kt + NS < nk; ++kt) stage = tile(kt, stage, true);
  for (; kt < nk; ++kt) stage = tile(kt, stage, false);
  }
#undef SLOTS
#undef SGB

  // ---- main loop, A K-contiguous: two wave groups in ping-pong -------------
  // Waves 0-3 (group 0) and 4-7 (group 1) sit one of each on every SIMD;
  // group g computes rows 128 g .. 128 g + 127 of the tile, so it alone reads
  // that half of the A tile, while both read the whole B tile.  LDS holds two
  // buffers for each A half (16 KiB) and three for B (32 KiB): 160 KiB.
  // Workgroup barriers cut time into phases of one K tile's MFMAs; in each
  // phase one group multiplies a K tile whose fragments it already holds
  // (64 MFMAs and nothing else, so nothing can hold them up) while the other
  // group reads the fragments of its next K tile out of LDS and issues the
  // loads.  Group 1 runs one phase behind:
  //   phase 2t:   group 0 reads tile t, loads;  group 1 multiplies tile t-1
  //   phase 2t+1: group 0 multiplies tile t;    group 1 reads tile t, loads
  // The loads of a read phase of tile t: the group's A half of tile t+1 (into
  // the A buffer of tile t-1) and the wave's half of its group's rows of B
  // tile t+2 (into the B buffer of tile t-1, which both groups have read by
  // then).  A wave waits for them at the end of its next MFMA phase, before
  // the barrier after which the first of them is read.  Issuing the loads
  // from the reading waves matters: an MFMA wave that issues a load while the
  // address unit is busy stalls its matrix core (measured: 4-7% slower).
  // Loads of tiles past the end of K read zeros into buffers no one reads
  // any more, so the in-flight counts are fixed.
  if constexpr (PP) {
    constexpr int ABUF = 128 * BK * 2, BBUF = 256 * BK * 2;
    constexpr int A0_OFF = 0, A1_OFF = 2 * ABUF, B_OFF = 4 * ABUF;
    static_assert(B_OFF + 3 * BBUF == PP_LDS, "two A-half buffers per group and three B buffers");
    constexpr int NQ = 4;   // loads per wave per K tile and operand stream
    const bool g0 = wave < 4;
    const int w4 = wave & 3;
    const int ah = wm, bh = g0 ? 1 : 0;
    // K-contiguous streams: wave w4 owns rows r0 + 32 w4 .. +31 of its
    // operand (r0 = 128 x its half); load q fills rows 8 q .. 8 q + 7 of
    // those, lane L taking row L/8 and LDS chunk L%8 = global chunk
    // (L%8) ^ swz(row), swz(row) = swz(8 (q & 1) + L/8).  One descriptor
    // bounds the 32 rows; the K offset is the scalar offset.
    const int lr = lane >> 3;
    const int a_r0 = ah * 128 + 32 * w4, b_r0 = bh * 128 + 32 * w4;
    auto a_rows_ptr = [&](int r0) -> const uint16_t* {
      if (PARTS && t->a_rows) {
        const int r = row0 + (r0 < rows ? r0 : 0);   // rows past the end: any part, size 0 below
        const int ab = r / t->a_rows;
        return t->a[ab] + (int64_t)(r - ab * t->a_rows) * p.lda;
      }
      return At + (int64_t)r0 * p.lda;
    };
    auto b_rows_ptr = [&](int r0, int kp) -> const uint16_t* {
      if (PARTS && t->b_nrows) {
        const int gb = grp * t->b_gstride;
        if (cols - r0 <= 0) return t->b[gb + kp];
        const int n = col0 + r0;
        const int nb = n / t->b_nrows;
        return t->b[gb + nb * t->b_nk + kp] + (int64_t)(n - nb * t->b_nrows) * p.ldb;
      }
      return Btile + (int64_t)r0 * p.ldb;
    };
    const uint32_t a_nrec = (uint32_t)(min(max(rows - a_r0, 0), 32) * p.lda * 2);
    const uint32_t b_nrec = (uint32_t)(min(max(cols - b_r0, 0), 32) * p.ldb * 2);
    const __amdgpu_buffer_rsrc_t rsa = make_rsrc(a_rows_ptr(a_r0), a_nrec);
    __amdgpu_buffer_rsrc_t rsb = make_rsrc(b_rows_ptr(b_r0, 0), b_nrec);
    uint32_t a_lo[2], b_lo[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      a_lo[e] = (uint32_t)(lr * p.lda * 2 + (((lane & 7) ^ swz(8 * e + lr)) << 4));
      b_lo[e] = (uint32_t)(lr * p.ldb * 2 + (((lane & 7) ^ swz(8 * e + lr)) << 4));
    }
    // MN-major B: wave w4 owns k rows 32 bh + 8 w4 .. +7; load q fills k rows
    // 2 q and 2 q + 1 of those, lane L taking row L/32 and LDS chunk L%32 =
    // global chunk (L%32) ^ 4 (row & 3).  A descriptor per K tile bounds the
    // rows at the end of K and the last row at the operand's last column.
    uint32_t b_mv[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int kr = 32 * bh + 8 * w4 + 2 * q + (lane >> 5);
      b_mv[q] = BMN ? (uint32_t)(kr * p.ldb * 2 + (((lane & 31) ^ mn_swz(kr)) << 4)) : 0u;
    }
    int b_kpart = 0;
    int b_kend = (PARTS && t->b_nrows) ? t->b_kcols : 0;
    struct LoadSet {
      __amdgpu_buffer_rsrc_t r;
      uint32_t so;
      uint32_t v[NQ];
      char* lds;
    };
    // K-contiguous chunk e-parity mask: chunks past the end of K read zero
    auto kmask = [&](int kb, int e) -> uint32_t {
      return (kb + (((lane & 7) ^ swz(8 * e + lr)) << 3) < k_end) ? 0u : OOB;
    };
    auto prep_a = [&](int kt, int buf) -> LoadSet {
      LoadSet L;
      const int kb = k_begin + kt * BK;
      L.r = rsa;
      L.so = (uint32_t)kb * 2;
      const uint32_t m0 = kmask(kb, 0), m1 = kmask(kb, 1);
#pragma unroll
      for (int q = 0; q < NQ; ++q) L.v[q] = (a_lo[q & 1] + (uint32_t)(q * 16 * p.lda)) | ((q & 1) ? m1 : m0);
      L.lds = smem + (ah ? A1_OFF : A0_OFF) + buf * ABUF + w4 * 4096;
      return L;
    };
    auto prep_b = [&](int kt, int buf) -> LoadSet {
      LoadSet L;
      const int kb = k_begin + kt * BK;
      L.lds = smem + B_OFF + buf * BBUF + bh * (BBUF / 2) + w4 * 4096;
      if constexpr (BMN) {
        const uint32_t kvalid = (uint32_t)min(max(k_end - kb, 0), BK);
        const uint32_t bytes = kvalid ? (uint32_t)(((int64_t)(kvalid - 1) * p.ldb + (p.N - col0)) * 2) : 0u;
        L.r = make_rsrc(Bg + (int64_t)kb * p.ldb + col0, bytes);
        L.so = 0;
#pragma unroll
        for (int q = 0; q < NQ; ++q) L.v[q] = b_mv[q];
        return L;
      }
      uint32_t so = (uint32_t)kb * 2;
      if (PARTS && t->b_nrows) {
        // the all_gather of B along K: K tiles never straddle a part (a tail
        // part may start several parts in); this wave's tiles come in order
        if (kb >= b_kend && b_kpart + 1 < t->b_nk) {
          while (kb >= b_kend && b_kpart + 1 < t->b_nk) {
            ++b_kpart;
            b_kend += t->b_kcols;
          }
          rsb = make_rsrc(b_rows_ptr(b_r0, b_kpart), b_nrec);
        }
        so = (uint32_t)(kb - (b_kend - t->b_kcols)) * 2;
      }
      L.r = rsb;
      L.so = so;
      const uint32_t m0 = kmask(kb, 0), m1 = kmask(kb, 1);
#pragma unroll
      for (int q = 0; q < NQ; ++q) L.v[q] = (b_lo[q & 1] + (uint32_t)(q * 16 * p.ldb)) | ((q & 1) ? m1 : m0);
      return L;
    };
    auto issue = [&](const LoadSet& L, int q) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(L.r, (lds_void*)(L.lds + q * 1024), 16, L.v[q], L.so, 0, 0);
    };
    auto issue_all = [&](const LoadSet& L) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) issue(L, q);
    };
    // fragments of k step ks of the tile in A buffer ai and B buffer bi
    auto ldfrag2 = [&](int ai, int bi, int ks, bf16x8* a, bf16x8* b) {
      const char* abuf = smem + (ah ? A1_OFF : A0_OFF) + ai * ABUF;
      const char* bbuf = smem + B_OFF + bi * BBUF;
      const int ko = ((4 * ks + g16) ^ fsw) << 4;
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] = *(const bf16x8*)(abuf + (i * 16 + (lane & 15)) * BK * 2 + ko);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        b[j] = BMN ? mn_frag(bbuf, ks, wn * 64 + j * 16)
                   : *(const bf16x8*)(bbuf + (wn * 64 + j * 16 + (lane & 15)) * BK * 2 + ko);
    };
    auto barrier = [] {
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_barrier" ::: "memory");
      __builtin_amdgcn_sched_barrier(0);
    };
    bf16x8 fa[KK][8], fb[KK][4];
    // prologue: this wave's A half of tile 0 and B half of tiles 0 and 1
    issue_all(prep_a(0, 0));
    issue_all(prep_b(0, 0));
    issue_all(prep_b(1, 1));
    WAIT_VMCNT(NQ);
    barrier();
    if (!g0) barrier();
    int ai = 0, bi = 0;   // buffers of tile kt: kt % 2, kt % 3
    for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) ldfrag2(ai, bi, kk, fa[kk], fb[kk]);
      // the group's A half of tile kt+1 (into the A buffer read two phases
      // ago) and its B half of tile kt+2 (into the B buffer of tile kt-1)
      const LoadSet LA = prep_a(kt + 1, ai ^ 1);
      const LoadSet LB = prep_b(kt + 2, bi == 0 ? 2 : bi - 1);
      issue_all(LA);
      issue_all(LB);
      WAIT_LGKMCNT(0);
      WAIT_VMCNT(2 * NQ);   // only the prologue's tile-1 loads can still be older
      barrier();
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) mma(fa[kk], fb[kk]);
      __builtin_amdgcn_sched_barrier(0);
      WAIT_VMCNT(0);   // this wave's loads of the read phase before
      barrier();
      ai ^= 1;
      bi = (bi == 2) ? 0 : bi + 1;
    }
    if (g0) barrier();
    WAIT_VMCNT(0);
    __syncthreads();   // every wave's loads landed and reads done: the buffers are free
    if (PHI_TAB) build_phi();
  }

  // ---- tail parts ----------------------------------------------------------------
  // Accumulator block acc[i][j] (4 floats) of thread tid is floats
  // 4 ((4 i + j) NT + tid) .. +3 of a part: float4 stores of consecutive threads.
  if constexpr (FIX) {
    const float* src = p.tail_ws + (size_t)blockIdx.x * p.tail_parts * (NT * 128);
    for (int q = 0; q < p.tail_parts; ++q) {   // ascending K
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 v = *(const f32x4*)(src + (size_t)q * (NT * 128) + ((i * 4 + j) * NT + tid) * 4);
          acc[i][j] = q ? acc[i][j] + v : v;
        }
    }
  } else if (tail_unit >= 0) {
    float* dst = p.tail_ws + (size_t)tail_unit * (NT * 128);
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) *(f32x4*)(dst + ((i * 4 + j) * NT + tid) * 4) = acc[i][j];
    return;
  }

  // ---- epilogue ----------------------------------------------------------------
  // Lane holds C[m][n..n+3] for each (i, j, g): 16-byte pieces of 32 rows per
  // store, which the memory system would see as partial lines.  The tile is
  // therefore staged through LDS and written back row by row, each row as
  // one contiguous run (bf16: 32 lanes x 16 B; fp32: 64 lanes x 16 B).
  // The output is stored non-temporally (streaming): every workgroup of a
  // wave stores its tile at the same moment, and the streaming stores drain
  // that burst faster (measured: 3.5% on bf16, 6-9% on fp32 outputs with a
  // 4096-long K loop).
  const float* bias = pick3(grp, p.bias[0], p.bias[1], p.bias[2]);
  void* Cg = pick3(grp, p.C[0], p.C[1], p.C[2]);
  __syncthreads();   // every wave is done with the K stages
  if (EPI == EPI_BF16 || EPI == EPI_BF16_SAVE) {
    uint16_t* cs = (uint16_t*)smem;
    auto stage = [&](bool apply_act) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int ml = wm * 128 + i * 16 + (lane & 15);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int nl = wn * 64 + j * 16 + 4 * g16;
            f32x4 v = acc[i][j];
            if (bias) {
              if (nl < cols) v += *(const f32x4*)(bias + col0 + nl);
            }
            if (ACT && apply_act) {
              const float2* tab = (const float2*)(smem + PHI_OFF);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float u = __builtin_amdgcn_fmed3f(__builtin_fmaf(v[e], PHI_SCALE, -PHI_LO * PHI_SCALE), 0.0f,
                                                        (float)PHI_N - 0.001f);
                const float fl = __builtin_floorf(u);
                const float2 pd = tab[(int)fl];
                v[e] *= __builtin_fmaf(u - fl, pd.y, pd.x);
              }
            }
            const bf16x4 o = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
            *(bf16x4*)(cs + ml * CPB + nl) = o;
        }
      }
    };
    // 16 rows per pass: thread t writes 8 columns (16 B) of row t / 32
    auto write = [&](uint16_t* out, bool parted) {
      const int cr = tid >> 5, cc = (tid & 31) * 8;
#pragma unroll 4
      for (int r0 = 0; r0 < BM; r0 += NT / 32) {
        const int r = r0 + cr;
        if (r >= rows || cc >= cols) continue;
        const i32x4 v = *(const i32x4*)(cs + r * CPB + cc);
        int64_t grow = row0 + r;
        uint16_t* ob = out;
        if (PARTS && parted) {   // the 16 rows of a pass share one part (c_rows % 16 == 0)
          const int cb = (row0 + r0) / t->c_rows;
          ob = (uint16_t*)t->c[cb];
          grow -= (int64_t)cb * t->c_rows;
        }
        uint16_t* dst = ob + grow * p.ldc + col0 + cc;
        if (cc + 8 <= cols) __builtin_nontemporal_store(v, (i32x4*)dst);
        else *(int2*)dst = make_int2(v[0], v[1]);   // a 4-column tail (cols % 8 == 4)
      }
    };
    if (EPI == EPI_BF16_SAVE) {   // the pre-activation first, for the backward pass
      stage(false);
      __syncthreads();
      write((uint16_t*)p.aux, false);
      __syncthreads();
    }
    stage(true);
    __syncthreads();
    write((uint16_t*)Cg, PARTS && t->c_rows);
  } else {
    // fp32 results (plain, residual or split partial): two halves of 128 rows.
    // Thread t writes 4 columns (16 B) of row t / 64 of each 8-row pass.  A
    // residual is read for all 16 passes of a half before the half is
    // staged, so the reads overlap the staging and are one round trip per
    // half rather than one per few passes (it may alias C: each element is
    // read and then written by the same thread).
    float* cs = (float*)smem;
    constexpr int NPASS = (BM / 2) / (NT / 64);
    const int cr = tid >> 6, cc = (tid & 63) * 4;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      f32x4 rv[NPASS];
      if (EPI == EPI_RESID_F32) {
#pragma unroll
        for (int k = 0; k < NPASS; ++k) {
          const int r0 = k * (NT / 64), r = q * (BM / 2) + r0 + cr;
          rv[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
          if (r < rows && cc < cols) {
            const int64_t m = row0 + r, n = col0 + cc;
            if (PARTS && t->c_rows) {   // into a part: the residual is the part itself
              const int cb = (row0 + q * (BM / 2) + r0) / t->c_rows;
              rv[k] = *(const f32x4*)((const float*)t->c[cb] + (m - (int64_t)cb * t->c_rows) * p.ldc + n);
            } else {
              rv[k] = *(const f32x4*)(p.resid + m * p.ldr + n);
            }
          }
        }
      }
      if (wm == q) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int ml = i * 16 + (lane & 15);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
              const int nl = wn * 64 + j * 16 + 4 * g16;
              f32x4 v = acc[i][j];
              if (EPI != EPI_PARTIAL) {
                if (bias) {
                  if (nl < cols) v += *(const f32x4*)(bias + col0 + nl);
                }
                if (ACT) {
#pragma unroll
                  for (int e = 0; e < 4; ++e) v[e] = gelu_erf(v[e]);
                }
              }
              *(f32x4*)(cs + ml * CPF + nl) = v;
          }
        }
      }
      __syncthreads();
#pragma unroll
      for (int k = 0; k < NPASS; ++k) {
        const int r0 = k * (NT / 64), rl = r0 + cr, r = q * (BM / 2) + rl;
        if (r >= rows || cc >= cols) continue;
        const f32x4 v = *(const f32x4*)(cs + rl * CPF + cc);
        const int64_t m = row0 + r, n = col0 + cc;
        if (EPI == EPI_PARTIAL) {
          *(f32x4*)(p.partial + split * p.part_stride + m * p.part_ld + n) = v;
        } else if (EPI == EPI_F32) {
          if (PARTS && t->c_rows) {   // the 8 rows of a pass share one part
            const int cb = (row0 + q * (BM / 2) + r0) / t->c_rows;
            __builtin_nontemporal_store(v, (f32x4*)((float*)t->c[cb] + (m - (int64_t)cb * t->c_rows) * p.ldc + n));
          } else {
            __builtin_nontemporal_store(v, (f32x4*)((float*)Cg + m * p.ldc + n));
          }
        } else if (PARTS && t->c_rows) {   // EPI_RESID_F32 into a part
          const int cb = (row0 + q * (BM / 2) + r0) / t->c_rows;
          __builtin_nontemporal_store(rv[k] + v, (f32x4*)((float*)t->c[cb] + (m - (int64_t)cb * t->c_rows) * p.ldc + n));
        } else {  // EPI_RESID_F32
          __builtin_nontemporal_store(rv[k] + v, (f32x4*)((float*)Cg + m * p.ldc + n));
        }
      }
      if (q == 0) __syncthreads();   // the second half reuses the buffer
    }
  }
}

template <int EPI, int ACT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_bf16_kernel(GemmParams p) { gemm_body<EPI, ACT, 0, 0>(p, nullptr); }

template <int EPI, int ACT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_bf16_parts_kernel(GemmParams p, GemmParts t) { gemm_body<EPI, ACT, 1, 0>(p, &t); }

template <int EPI, int ACT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_bf16_fixup_kernel(GemmParams p) { gemm_body<EPI, ACT, 0, 1>(p, nullptr); }

template <int EPI, int ACT, int AMN, int BMN>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_bf16_mn_kernel(GemmParams p) { gemm_body<EPI, ACT, 0, 0, AMN, BMN>(p, nullptr); }

template <int EPI, int ACT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_bf16_parts_fixup_kernel(GemmParams p, GemmParts t) { gemm_body<EPI, ACT, 1, 1>(p, &t); }

// Workgroups of the main launch: every tile once, or the whole tiles plus
// tail_parts per tail tile.
int64_t main_grid(const GemmParams& p) {
  const int64_t ntiles = (int64_t)p.tiles_m * p.tiles_n;
  if (p.tail_parts > 1) return p.tail_base + (ntiles - p.tail_base) * p.tail_parts;
  return ntiles * p.nsplit;
}

// The tail split's invariants: whole-K accumulation otherwise, every part at
// least one K tile, a workspace to hold the parts.
bool tail_ok(const GemmParams& p) {
  const int64_t ntiles = (int64_t)p.tiles_m * p.tiles_n;
  const int64_t nk = (p.K + BK - 1) / BK;
  return p.nsplit == 1 && p.tail_ws && p.tail_base >= 0 && p.tail_base < ntiles && p.tail_kt > 0 &&
         (int64_t)(p.tail_parts - 1) * p.tail_kt < nk;
}

template <int EPI, int ACT, int FIX>
hipError_t launch(const GemmParams& p, hipStream_t s) {
  if (p.tail_parts > 1 && !tail_ok(p)) return hipErrorInvalidValue;
  if (FIX) {
    if (p.tail_parts <= 1) return hipErrorInvalidValue;
    const int64_t nwg = (int64_t)p.tiles_m * p.tiles_n - p.tail_base;
    hipLaunchKernelGGL((gemm_bf16_fixup_kernel<EPI, ACT>), dim3((unsigned)nwg), dim3(NT), 0, s, p);
  } else {
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI, ACT>), dim3((unsigned)main_grid(p)), dim3(NT), 0, s, p);
  }
  return hipGetLastError();
}

template <int EPI, int ACT, int FIX>
hipError_t launch_parts(const GemmParams& p, const GemmParts& t, hipStream_t s) {
  if (p.tail_parts > 1 && !tail_ok(p)) return hipErrorInvalidValue;
  if (FIX) {
    if (p.tail_parts <= 1) return hipErrorInvalidValue;
    const int64_t nwg = (int64_t)p.tiles_m * p.tiles_n - p.tail_base;
    hipLaunchKernelGGL((gemm_bf16_parts_fixup_kernel<EPI, ACT>), dim3((unsigned)nwg), dim3(NT), 0, s, p, t);
  } else {
    hipLaunchKernelGGL((gemm_bf16_parts_kernel<EPI, ACT>), dim3((unsigned)main_grid(p)), dim3(NT), 0, s, p, t);
  }
  return hipGetLastError();
}

template <int EPI, int ACT, int AMN, int BMN>
hipError_t launch_mn(const GemmParams& p, hipStream_t s) {
  if (p.tail_parts > 1 && !tail_ok(p)) return hipErrorInvalidValue;
  hipLaunchKernelGGL((gemm_bf16_mn_kernel<EPI, ACT, AMN, BMN>), dim3((unsigned)main_grid(p)), dim3(NT), 0, s, p);
  return hipGetLastError();
}

// MN-major operands; the fixup launch is the common one.  An activation (and
// the kept pre-activation) only with A K-contiguous and B stored [K, N]: the
// forward products of the blocks, whose weights are [fan_in, fan_out].
template <int AMN, int BMN>
hipError_t dispatch_mn(const GemmParams& p, hipStream_t s) {
  if constexpr (AMN == 0 && BMN == 1) {
    switch (p.epi * 2 + (p.act ? 1 : 0)) {
      case EPI_BF16 * 2 + 0: return launch_mn<EPI_BF16, 0, 0, 1>(p, s);
      case EPI_BF16 * 2 + 1: return launch_mn<EPI_BF16, 1, 0, 1>(p, s);
      case EPI_F32 * 2 + 0: return launch_mn<EPI_F32, 0, 0, 1>(p, s);
      case EPI_F32 * 2 + 1: return launch_mn<EPI_F32, 1, 0, 1>(p, s);
      case EPI_PARTIAL * 2 + 0: return launch_mn<EPI_PARTIAL, 0, 0, 1>(p, s);
      case EPI_RESID_F32 * 2 + 0: return launch_mn<EPI_RESID_F32, 0, 0, 1>(p, s);
      case EPI_BF16_SAVE * 2 + 0: return launch_mn<EPI_BF16_SAVE, 0, 0, 1>(p, s);
      case EPI_BF16_SAVE * 2 + 1: return launch_mn<EPI_BF16_SAVE, 1, 0, 1>(p, s);
      default: return hipErrorInvalidValue;
    }
  } else {
    if (p.act) return hipErrorInvalidValue;
    switch (p.epi) {
      case EPI_BF16: return launch_mn<EPI_BF16, 0, AMN, BMN>(p, s);
      case EPI_F32: return launch_mn<EPI_F32, 0, AMN, BMN>(p, s);
      case EPI_PARTIAL: return launch_mn<EPI_PARTIAL, 0, AMN, BMN>(p, s);
      case EPI_RESID_F32: return launch_mn<EPI_RESID_F32, 0, AMN, BMN>(p, s);
      default: return hipErrorInvalidValue;
    }
  }
}

template <int FIX>
hipError_t dispatch(const GemmParams& p, hipStream_t s) {
  if (!FIX && (p.a_mn || p.b_mn)) {
    if (p.a_mn && p.b_mn) return dispatch_mn<1, 1>(p, s);
    return p.a_mn ? dispatch_mn<1, 0>(p, s) : dispatch_mn<0, 1>(p, s);
  }
  switch (p.epi * 2 + (p.act ? 1 : 0)) {
    case EPI_BF16 * 2 + 0: return launch<EPI_BF16, 0, FIX>(p, s);
    case EPI_BF16 * 2 + 1: return launch<EPI_BF16, 1, FIX>(p, s);
    case EPI_F32 * 2 + 0: return launch<EPI_F32, 0, FIX>(p, s);
    case EPI_F32 * 2 + 1: return launch<EPI_F32, 1, FIX>(p, s);
    case EPI_PARTIAL * 2 + 0: return FIX ? hipErrorInvalidValue : launch<EPI_PARTIAL, 0, 0>(p, s);
    case EPI_RESID_F32 * 2 + 0: return launch<EPI_RESID_F32, 0, FIX>(p, s);
    case EPI_RESID_F32 * 2 + 1: return launch<EPI_RESID_F32, 1, FIX>(p, s);
    case EPI_BF16_SAVE * 2 + 0: return launch<EPI_BF16_SAVE, 0, FIX>(p, s);
    case EPI_BF16_SAVE * 2 + 1: return launch<EPI_BF16_SAVE, 1, FIX>(p, s);
    default: return hipErrorInvalidValue;
  }
}

template <int FIX>
hipError_t dispatch_parts(const GemmParams& p, const GemmParts& t, hipStream_t s) {
  // device-local arrays: whole-K accumulation only (a split partial has no
  // owner), K-contiguous operands
  if (p.nsplit != 1 || p.a_mn || p.b_mn || (t.a_rows && t.a_rows % 64) || (t.c_rows && t.c_rows % 16) ||
      (t.b_nrows && (t.b_nrows % 64 || t.b_kcols % 64 || t.b_nk < 1 || t.b_gstride < 0 ||
                     (p.ngroups > 1 && t.b_gstride == 0) ||
                     (int64_t)(p.ngroups - 1) * t.b_gstride + (int64_t)((p.N + t.b_nrows - 1) / t.b_nrows) * t.b_nk > kMaxParts)))
    return hipErrorInvalidValue;
  switch (p.epi * 2 + (p.act ? 1 : 0)) {
    case EPI_BF16 * 2 + 0: return launch_parts<EPI_BF16, 0, FIX>(p, t, s);
    case EPI_BF16 * 2 + 1: return launch_parts<EPI_BF16, 1, FIX>(p, t, s);
    case EPI_F32 * 2 + 0: return launch_parts<EPI_F32, 0, FIX>(p, t, s);
    case EPI_RESID_F32 * 2 + 0: return launch_parts<EPI_RESID_F32, 0, FIX>(p, t, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int gemm_bf16_tile_m() { return BM; }
int gemm_bf16_tile_n() { return BN; }

hipError_t launch_gemm_bf16(const GemmParams& p, hipStream_t s) { return dispatch<0>(p, s); }
hipError_t launch_gemm_bf16_fixup(const GemmParams& p, hipStream_t s) { return dispatch<1>(p, s); }
hipError_t launch_gemm_bf16_parts(const GemmParams& p, const GemmParts& t, hipStream_t s) {
  return dispatch_parts<0>(p, t, s);
}
hipError_t launch_gemm_bf16_parts_fixup(const GemmParams& p, const GemmParts& t, hipStream_t s) {
  return dispatch_parts<1>(p, t, s);
}

}  // namespace partir
