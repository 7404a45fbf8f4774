// Softmax attention backward for gfx950, d_head = 128, bf16 in / bf16 out.
//
// Given Q, K, V, the forward output O, its cotangent dO and the per-row
// log-sum-exp of the scaled scores (base 2: lse2 = log2 sum_j 2^(c s_j),
// c = scale log2 e), with P = 2^(c S - lse2):
//     D  = rowsum(dO * O)             dV = P^T dO        dP = dO V^T
//     dS = P * (dP - D)               dQ = scale dS K    dK = scale dS^T Q
// Two passes, each a loop over one axis of the score matrix with the other
// axis held in registers, so every gradient is accumulated by one workgroup
// in a fixed order (no atomics: deterministic):
//  * dq pass: workgroup = (sequence, head, 128 queries), 4 waves x 32
//    queries; keys stream through LDS 64 at a time.  S^T = K Q^T and
//    dP^T = V dO^T put one query per lane, dQ^T += K^T dS^T per 32 keys
//    (K^T read with ds_read_b64_tr_b16).  It also writes D for the second
//    pass.
//  * dv and dk passes: workgroup = (sequence, head, 128 keys), 4 waves x 32
//    keys; queries stream 64 at a time.  S = Q K^T and dP = dO V^T put one
//    key per lane, dV^T += dO^T P (dv pass) and dK^T += Q^T dS (dk pass),
//    from transposed reads of the dO and Q tiles.
// Inside a 16-wide MFMA contraction step the order of the contracted
// positions is permuted identically on both operands (exact for a sum).
// All LDS tiles are 64 rows x 256 B with 16-byte chunks XOR-swizzled by row
// (swz), so that both the row reads and the transposed reads hit every bank
// once.  The causal mask costs VALU work only on blocks that cross a wave's
// diagonal, and the block loops run two blocks per trip so that the LDS stage
// of each is a constant (its offset folds into the LDS instructions).
#include <type_traits>

#include "kernels.h"
#include "lds_dma.h"

namespace partir {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int DH = 128, NT = 256;
constexpr int TR = 64;                 // rows of a streamed tile
constexpr int TP = 256;                // tile row pitch (bytes)
constexpr int TILE = TR * TP;          // 16 KiB

// The XOR applied to the 16-byte chunk index of a tile row: row 4 b + a of a
// 16-row group (a, b < 4) gets 4 a + b.  A row read (16 lanes on 16
// consecutive rows, one logical chunk) lands on 16 distinct chunks; half a
// transposed read (4 consecutive rows x one aligned 64-byte group) does too,
// since the row's low two bits move it to another 64-byte group.  (XOR with
// the row's low four bits, which serves the row reads alone, put the four
// rows of a transposed read on the same 16 banks.)
__device__ __forceinline__ int swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

// byte offset of (row, byte column) in a swizzled tile
__device__ __forceinline__ int toff(int row, int colb) {
  return row * TP + (((colb >> 4) ^ swz(row)) << 4) + (colb & 15);
}

// two fp32 values rounded to bf16 into elements i, i + 1 of x (one
// v_cvt_pk_bf16_f32)
__device__ __forceinline__ void put2(bf16x8& x, int i, float a, float b) {
  const f32x2 f = {a, b};
  const bf16x2 r = __builtin_convertvector(f, bf16x2);
  x[i] = r[0];
  x[i + 1] = r[1];
}


// Streams two [64 x 128] bf16 tiles (rows of X and Y, head columns) into a
// swizzled LDS stage with buffer loads that write LDS directly: load j of
// wave w fills tile rows 16 j + 4 w .. +4 (1 KiB, lane L at byte 16 L), so
// lane L reads the global chunk that belongs at its LDS position,
// (L % 16) ^ swz(row), which does not depend on j (the row step enters as a
// scalar offset).
struct TileDma {
  __amdgpu_buffer_rsrc_t rx, ry;
  uint32_t vx, vy;           // per-lane byte offsets of load 0
  uint32_t stepx, stepy;     // bytes per 64-row tile
  uint32_t jx, jy;           // bytes per 16 rows
  int w;
  __device__ void init(const uint16_t* X, int64_t ldx, const uint16_t* Y, int64_t ldy, int S, int tid) {
    w = tid >> 6;
    const int lane = tid & 63;
    const int row = 4 * w + (lane >> 4);
    const int chunk = (lane & 15) ^ swz(row);
    rx = make_rsrc(X, (uint32_t)((S - 1) * ldx * 2 + DH * 2));
    ry = make_rsrc(Y, (uint32_t)((S - 1) * ldy * 2 + DH * 2));
    vx = (uint32_t)(row * ldx * 2 + chunk * 16);
    vy = (uint32_t)(row * ldy * 2 + chunk * 16);
    stepx = (uint32_t)(TR * ldx * 2);
    stepy = (uint32_t)(TR * ldy * 2);
    jx = (uint32_t)(16 * ldx * 2);
    jy = (uint32_t)(16 * ldy * 2);
  }
  // tile `blk` into the LDS tiles tx, ty (8 loads per wave in flight after)
  __device__ void load(int blk, char* tx, char* ty) const {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)(tx + j * 4096 + w * 1024), 16, vx,
                                               (uint32_t)blk * stepx + j * jx, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, (lds_void*)(ty + j * 4096 + w * 1024), 16, vy,
                                               (uint32_t)blk * stepy + j * jy, 0, 0);
    }
  }
};

// A operand of a 32-row MFMA block read row-wise from a tile: rows r0 + (lane
// & 31), contraction (d) chunk 2 ds + h.
__device__ __forceinline__ bf16x8 row_frag(const char* tile, int r0, int col, int h, int ds) {
  return *(const bf16x8*)(tile + toff(r0 + col, (2 * ds + h) * 16));
}

// A operand X^T[d rows 32 dt.., positions 16 u..] of a tile X [positions x d],
// the positions permuted as the score registers are (see the forward kernel).
__device__ __forceinline__ bf16x8 tr_frag(const char* tile, int u, int dt, int v_row, int v_colb) {
  const int row = 16 * u + v_row, colb = 64 * dt + v_colb;
  const i16x4 lo = lds_read_tr16(tile + toff(row, colb));
  const i16x4 hi = lds_read_tr16(tile + toff(row + 8, colb));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ void zero(f32x16& a) {
#pragma unroll
  for (int v = 0; v < 16; ++v) a[v] = 0.0f;
}

// ---------------------------------------------------------------------------
// dq pass
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attention_bwd_dq_kernel(AttnBwdParams p) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * 2 * TILE];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, col = lane & 31;

  const int nqb = p.S / 128;
  const int nbh = p.B * p.H;
  const int qb = nqb - 1 - (int)(blockIdx.x / nbh);   // heaviest query blocks first
  const int bh = blockIdx.x % nbh;
  const int b = bh / p.H, head = bh - b * p.H;
  const int q0 = qb * 128;
  const int64_t tok0 = (int64_t)b * p.S;
  const int qi = q0 + 32 * w + col;
  const int64_t tq = tok0 + qi;

  // Q and dO of this lane's query (B operands), D = rowsum(dO * O)
  bf16x8 qf[8], gf[8];
  float dsum = 0.0f;
  {
    const uint16_t* qrow = p.Q + tq * p.ldq + head * DH + 8 * h;
    const uint16_t* grow = p.dO + tq * p.ldg + head * DH + 8 * h;
    const uint16_t* orow = p.O + tq * p.ldo + head * DH + 8 * h;
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) {
      qf[ds] = *(const bf16x8*)(qrow + 16 * ds);
      gf[ds] = *(const bf16x8*)(grow + 16 * ds);
      const bf16x8 of = *(const bf16x8*)(orow + 16 * ds);
#pragma unroll
      for (int e = 0; e < 8; ++e) dsum += (float)gf[ds][e] * (float)of[e];
    }
  }
  const float Dq = dsum + __shfl_xor(dsum, 32);
  const float lse = p.lse[tq * p.H + head];
  if (h == 0) p.Dstat[tq * p.H + head] = Dq;

  TileDma kv;
  kv.init(p.K + tok0 * p.ldk + head * DH, p.ldk, p.V + tok0 * p.ldv + head * DH, p.ldv, p.S, tid);

  const int j16 = lane & 15, G = lane >> 4, hh = G >> 1;
  const int v_row = 4 * hh + (j16 >> 2);
  const int v_colb = 2 * (16 * (G & 1) + 4 * (j16 & 3));

  f32x16 dq[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) zero(dq[d]);

  const int nkb = p.causal ? (q0 + 128) / TR : p.S / TR;
  const int wave_last_q = q0 + 32 * w + 31;
  const float c = p.scale_log2;
  // Key block kb from LDS stage `stage`, block kb + 1 streaming into the
  // other stage (last read in the previous iteration, before its barrier).
  auto iter = [&](int kb, auto stage) {
    const int cur = stage;
    if (kb + 1 < nkb) kv.load(kb + 1, smem + (cur ^ 1) * 2 * TILE, smem + (cur ^ 1) * 2 * TILE + TILE);
    const int k0 = kb * TR;
    if (!p.causal || k0 <= wave_last_q) {
      const char* ks = smem + cur * 2 * TILE;
      const char* vs = ks + TILE;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        if (p.causal && k0 + 32 * t > wave_last_q) continue;   // wave-uniform: every key follows every query
        f32x16 s, dp;
        zero(s);
        zero(dp);
#pragma unroll
        for (int ds = 0; ds < 8; ++ds) {
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(ks, 32 * t, col, h, ds), qf[ds], s, 0, 0, 0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(vs, 32 * t, col, h, ds), gf[ds], dp, 0, 0, 0);
        }
        float pr[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) pr[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c, -lse));
        if (p.causal && k0 + 32 * t + 31 > q0 + 32 * w) {   // wave-uniform: keys past some query
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (k0 + 32 * t + 8 * (v >> 2) + 4 * h + (v & 3) > qi) pr[v] = 0.0f;
        }
        bf16x8 dsf[2];
#pragma unroll
        for (int v = 0; v < 16; v += 2)
          put2(dsf[v >> 3], v & 7, pr[v] * (dp[v] - Dq), pr[v + 1] * (dp[v + 1] - Dq));
        // dQ^T += K^T dS^T over these 32 keys, 2 steps of 16
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int d = 0; d < 4; ++d)
            dq[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag(ks, 2 * t + uu, d, v_row, v_colb), dsf[uu], dq[d], 0,
                                                            0, 0);
      }
    }
    WAIT_VMCNT(0);
    __syncthreads();
  };
  kv.load(0, smem, smem + TILE);
  WAIT_VMCNT(0);
  __syncthreads();
  for (int kb = 0; kb < nkb; kb += 2) {
    iter(kb, std::integral_constant<int, 0>{});
    if (kb + 1 < nkb) iter(kb + 1, std::integral_constant<int, 1>{});
  }

  // dQ[query][d] = scale * dQ^T: lane holds rows d = 32 dt + 8 (v>>2) + 4 h + (v&3)
  uint16_t* out = p.dQ + tq * p.lddq + head * DH;
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const bf16x4 o = {(__bf16)(dq[d][4 * g + 0] * p.scale), (__bf16)(dq[d][4 * g + 1] * p.scale),
                        (__bf16)(dq[d][4 * g + 2] * p.scale), (__bf16)(dq[d][4 * g + 3] * p.scale)};
      *(bf16x4*)(out + 32 * d + 8 * g + 4 * h) = o;
    }
}

// ---------------------------------------------------------------------------
// dkv pass
// ---------------------------------------------------------------------------
// MODE 1: dV (S recomputed, dV^T += dO^T P); MODE 2: dK (S and dP
// recomputed, dK^T += Q^T dS).  One pass doing both needs 287 registers
// (one wave per SIMD); the two passes recompute S once more but fit two
// waves per SIMD, which more than pays (0.84 -> 0.74 ms for the whole
// backward at 4 x 2048 tokens, 32 heads, when it was measured).
template <int MODE>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attention_bwd_dkv_kernel(AttnBwdParams p) {
  constexpr bool DO_V = MODE == 1, DO_K = MODE == 2;
  __shared__ __attribute__((aligned(1024))) char smem[2 * 2 * TILE];
  __shared__ float stat[2][2][TR];   // [stage][-lse2 / c, -D][query]
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, col = lane & 31;

  const int nbh = p.B * p.H;
  const int kblk = (int)(blockIdx.x / nbh);          // earliest key blocks (most queries) first
  const int bh = blockIdx.x % nbh;
  const int b = bh / p.H, head = bh - b * p.H;
  const int k0 = kblk * 128;
  const int64_t tok0 = (int64_t)b * p.S;
  const int kj = k0 + 32 * w + col;                  // this lane's key
  const int64_t tk = tok0 + kj;

  bf16x8 kf[8], vf[8];
  {
    const uint16_t* krow = p.K + tk * p.ldk + head * DH + 8 * h;
    const uint16_t* vrow = p.V + tk * p.ldv + head * DH + 8 * h;
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) {
      kf[ds] = *(const bf16x8*)(krow + 16 * ds);
      if (DO_K) vf[ds] = *(const bf16x8*)(vrow + 16 * ds);
    }
  }

  TileDma qg;
  qg.init(p.Q + tok0 * p.ldq + head * DH, p.ldq, p.dO + tok0 * p.ldg + head * DH, p.ldg, p.S, tid);
  float st_l = 0.0f, st_d = 0.0f;
  const float inv_c = 1.0f / p.scale_log2;
  auto sload = [&](int blk) {
    if (tid < TR) {
      const int64_t t = tok0 + (int64_t)blk * TR + tid;
      st_l = p.lse[t * p.H + head];
      if (DO_K) st_d = p.Dstat[t * p.H + head];
    }
  };
  auto sstore = [&](int buf) {
    if (tid < TR) {
      stat[buf][0][tid] = -st_l * inv_c;
      stat[buf][1][tid] = -st_d;
    }
  };

  const int j16 = lane & 15, G = lane >> 4, hh = G >> 1;
  const int v_row = 4 * hh + (j16 >> 2);
  const int v_colb = 2 * (16 * (G & 1) + 4 * (j16 & 3));

  f32x16 dk[4], dv[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    zero(dk[d]);
    zero(dv[d]);
  }

  const int qb_begin = p.causal ? k0 / TR : 0;
  const int nqb = p.S / TR;
  const int wave_first_k = k0 + 32 * w;
  const float c = p.scale_log2;
  // Query block qb from LDS stage `stage`, block qb + 1 and its statistics
  // streaming into the other stage (last read in the previous iteration,
  // before its barrier).
  auto iter = [&](int qb, auto stage) {
    const int cur = stage;
    if (qb + 1 < nqb) {
      qg.load(qb + 1, smem + (cur ^ 1) * 2 * TILE, smem + (cur ^ 1) * 2 * TILE + TILE);
      sload(qb + 1);
    }
    const int q0 = qb * TR;
    if (!p.causal || q0 + TR - 1 >= wave_first_k) {
      const char* qs = smem + cur * 2 * TILE;
      const char* gs = qs + TILE;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        if (p.causal && q0 + 32 * t + 31 < wave_first_k) continue;   // wave-uniform: sees none of these keys
        // The accumulators start at -lse2 / c and -D of their rows (queries),
        // so S - lse2 / c and dP - D come out of the products.
        f32x16 s, dp;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x4 l4 = *(const f32x4*)&stat[cur][0][32 * t + 8 * i + 4 * h];
#pragma unroll
          for (int j = 0; j < 4; ++j) s[4 * i + j] = l4[j];
          if (DO_K) {
            const f32x4 d4 = *(const f32x4*)&stat[cur][1][32 * t + 8 * i + 4 * h];
#pragma unroll
            for (int j = 0; j < 4; ++j) dp[4 * i + j] = d4[j];
          }
        }
#pragma unroll
        for (int ds = 0; ds < 8; ++ds) {
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(qs, 32 * t, col, h, ds), kf[ds], s, 0, 0, 0);
          if (DO_K)
            dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(gs, 32 * t, col, h, ds), vf[ds], dp, 0, 0, 0);
        }
        // lane: key kj; element v: query q0 + 32 t + 8 (v>>2) + 4 h + (v&3)
        float pr[16];
#pragma unroll
        for (int v = 0; v < 16; ++v)
          pr[v] = __builtin_amdgcn_exp2f(s[v] * c);
        if (p.causal && q0 + 32 * t < wave_first_k + 31) {   // wave-uniform: queries before some key
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (q0 + 32 * t + 8 * (v >> 2) + 4 * h + (v & 3) < kj) pr[v] = 0.0f;
        }
        bf16x8 pf[2], dsf[2];
#pragma unroll
        for (int v = 0; v < 16; v += 2) {
          if (DO_V) put2(pf[v >> 3], v & 7, pr[v], pr[v + 1]);
          if (DO_K) put2(dsf[v >> 3], v & 7, pr[v] * dp[v], pr[v + 1] * dp[v + 1]);
        }
        // dV^T += dO^T P and dK^T += Q^T dS over these 32 queries (2 steps of 16)
#pragma unroll
        for (int uu = 0; uu < 2; ++uu) {
          const int u = 2 * t + uu;
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            if (DO_V)
              dv[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag(gs, u, d, v_row, v_colb), pf[uu], dv[d], 0, 0, 0);
            if (DO_K)
              dk[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag(qs, u, d, v_row, v_colb), dsf[uu], dk[d], 0, 0, 0);
          }
        }
      }
    }
    if (qb + 1 < nqb) sstore(cur ^ 1);
    WAIT_VMCNT(0);
    __syncthreads();
  };
  qg.load(qb_begin, smem, smem + TILE);
  sload(qb_begin);
  sstore(0);
  WAIT_VMCNT(0);
  __syncthreads();
  for (int qb = qb_begin; qb < nqb; qb += 2) {
    iter(qb, std::integral_constant<int, 0>{});
    if (qb + 1 < nqb) iter(qb + 1, std::integral_constant<int, 1>{});
  }

  uint16_t* okr = p.dK + tk * p.lddk + head * DH;
  uint16_t* ovr = p.dV + tk * p.lddv + head * DH;
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      if (DO_K) {
        const bf16x4 ko = {(__bf16)(dk[d][4 * g + 0] * p.scale), (__bf16)(dk[d][4 * g + 1] * p.scale),
                           (__bf16)(dk[d][4 * g + 2] * p.scale), (__bf16)(dk[d][4 * g + 3] * p.scale)};
        *(bf16x4*)(okr + 32 * d + 8 * g + 4 * h) = ko;
      }
      if (DO_V) {
        const bf16x4 vo = {(__bf16)dv[d][4 * g + 0], (__bf16)dv[d][4 * g + 1], (__bf16)dv[d][4 * g + 2],
                           (__bf16)dv[d][4 * g + 3]};
        *(bf16x4*)(ovr + 32 * d + 8 * g + 4 * h) = vo;
      }
    }
}

}  // namespace

hipError_t launch_attention_backward(const AttnBwdParams& p, hipStream_t s) {
  if (p.B == 0 || p.S == 0 || p.H == 0) return hipSuccess;
  if (p.S % 128) return hipErrorInvalidValue;
  const unsigned nwg = (unsigned)(p.S / 128) * p.B * p.H;
  hipLaunchKernelGGL(attention_bwd_dq_kernel, dim3(nwg), dim3(NT), 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attention_bwd_dkv_kernel<1>, dim3(nwg), dim3(NT), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attention_bwd_dkv_kernel<2>, dim3(nwg), dim3(NT), 0, s, p);
  return hipGetLastError();
}

}  // namespace partir
