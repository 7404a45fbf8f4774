// Softmax attention forward for gfx950, d_head = 128, bf16 in / bf16 out.
//
// One workgroup = one (sequence, head, 128-query block); four waves own 32
// queries each.  Keys and values stream through a double-buffered LDS stage
// BKV = 32 (or 64) keys at a time.  Per key block each wave computes
//     S^T[BKV keys x 32 queries] = K_blk . Q^T      (v_mfma_f32_32x32x16_bf16)
// so that every lane owns one query column: the running max and sum of the
// online softmax are per-lane registers, and exp(S^T - max) converted to bf16
// is directly the B operand of
//     O^T[128 d x 32 queries] += V_blk^T . P^T
// The V^T operand is read from the row-major V tile with ds_read_b64_tr_b16;
// the key order inside each 16-key MFMA step is permuted identically on the P
// and V sides (any order is exact for the contraction).
// With causal masking a query sees keys at positions <= its own.
#include <type_traits>

#include "kernels.h"
#include "lds_dma.h"

namespace partir {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int DH = 128, BQ = 128, NT = 256;
// K and V tiles: BKV rows of 256 B, written by direct-to-LDS buffer loads
// (each wave load fills 1 KiB = 4 whole rows).  K: 16-byte chunk c of row r
// at position c ^ (r & 15), so the 32 rows one S^T fragment read touches hit
// all 64 banks.  V: 64-byte group g of row r at position g ^ (r & 3), so the
// 4 rows x 64 B one half of a ds_read_b64_tr_b16 touches hit all 64 banks.
constexpr int RP = 256;

// LDS reads of K fragments through a restrict pointer, for the same reason
// as lds_read_tr16: the alias scope keeps the wait insertion from making them
// wait on the next tiles' DMA (which writes the other stage).
__device__ __forceinline__ bf16x8 lds_read_b128(const char* __restrict__ p) { return *(const bf16x8*)p; }

// BKV = 32: three workgroups per CU (32 KiB of LDS each, at most 168
// VGPRs); the third wave per SIMD hides more of the load, LDS and barrier
// waits than the halved work between barriers costs.  BKV = 64: two per CU
// (64 KiB), fewer barriers; the host takes it for grids smaller than the
// CU count, where occupancy cannot help.
template <int BKV>
__global__ __launch_bounds__(NT, BKV == 32 ? 3 : 2)
void attention_kernel(AttnParams p) {
  static_assert(BKV == 32 || BKV == 64, "key blocks of 32 or 64");
  constexpr int NSUB = BKV / 32;            // 32-key sub-tiles of S^T
  constexpr int T_BYTES = BKV * RP;
  constexpr int STAGE = 2 * T_BYTES;      // K tile, then V tile
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, so per-wave tests branch
  const int h = lane >> 5, col = lane & 31;

  // heaviest (latest) query blocks first: causal work grows with the block
  // index; with a split key axis, the shards of one query block are adjacent
  const int nqb = p.S / BQ;
  const int nbh = p.B * p.H;
  const int per_qb = nbh * p.nsplit;
  // Workgroup i runs on XCD i mod 8.
  int qs, split, bh;
  if (p.nsplit == 1 && (nbh & 7) == 0) {
    // Unsplit: XCD x takes (sequence, head)s x, x + 8, ... in groups of up
    // to 8, each group's query blocks heaviest first, so the workgroups an
    // XCD holds at once stream the same few heads' K / V through its L2.
    const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
    int G = 8;
    while ((nbh / 8) % G) G >>= 1;
    const int gen = j / (G * nqb), r = j - gen * (G * nqb);
    qs = r / G;
    bh = (gen * G + (r - qs * G)) * 8 + x;
    split = 0;
  } else {
    // Under a causal mask the shards of early keys carry most of the work,
    // so (shard, head) must not stay tied to one XCD: rotating it by the
    // query block spreads every shard over all XCDs.
    qs = blockIdx.x / per_qb;
    int inner = blockIdx.x - qs * per_qb;
    if (p.nsplit > 1) inner = (inner + qs) % per_qb;
    split = inner / nbh;
    bh = inner - split * nbh;
  }
  const int qb = nqb - 1 - qs;
  const int b = bh / p.H, head = bh - b * p.H;
  const int q0 = qb * BQ;
  const int64_t tok0 = (int64_t)b * p.S;
  // causal: a key shard that starts past this query block's last query holds
  // nothing for it; the combine does not read such a shard, so it is skipped
  // (workgroup-uniform, before any barrier)
  if (p.nsplit > 1 && p.causal && split * p.kb_per * 64 > q0 + BQ - 1) return;

  // ---- this lane's query fragments (B operand of S^T = K Q^T), kept in VGPRs
  const int qi = q0 + 32 * w + col;      // query position of this lane's column
  bf16x8 qf[8];
  {
    const uint16_t* qrow = p.Q + (tok0 + qi) * p.ldq + head * DH + 8 * h;
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) qf[ds] = *(const bf16x8*)(qrow + 16 * ds);
  }

  // ---- K / V tile loads straight into LDS: wave load i of wave w fills rows
  // 16 i + 4 w .. +3 of a tile; lane L writes LDS chunk L % 16 of row
  // 16 i + 4 w + L / 16, so it reads the global chunk that the tile's swizzle
  // puts there.  The key block and the row block i enter as scalar offsets.
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(p.K + tok0 * p.ldk + head * DH, (uint32_t)((p.S - 1) * p.ldk * 2 + DH * 2));
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(p.V + tok0 * p.ldv + head * DH, (uint32_t)((p.S - 1) * p.ldv * 2 + DH * 2));
  const int lrow = 4 * w + (lane >> 4), lch = lane & 15;   // row within a 16-row block; LDS chunk
  const uint32_t kvo = (uint32_t)(lrow * p.ldk * 2 + ((lch ^ (lrow & 15)) << 4));
  const uint32_t vvo = (uint32_t)(lrow * p.ldv * 2 + ((((lch >> 2) ^ (lrow & 3)) << 2 | (lch & 3)) << 4));
  const uint32_t kstep = (uint32_t)(BKV * p.ldk * 2), vstep = (uint32_t)(BKV * p.ldv * 2);
  const uint32_t krow16 = (uint32_t)(16 * p.ldk * 2), vrow16 = (uint32_t)(16 * p.ldv * 2);
  auto gload = [&](int kb, int buf) {
    char* ks = smem + buf * STAGE + w * 1024;
    char* vs = ks + T_BYTES;
#pragma unroll
    for (int i = 0; i < BKV / 16; ++i) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(krs, (lds_void*)(ks + i * 4096), 16, kvo,
                                               (uint32_t)kb * kstep + i * krow16, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vrs, (lds_void*)(vs + i * 4096), 16, vvo,
                                               (uint32_t)kb * vstep + i * vrow16, 0, 0);
    }
  };

  f32x16 oacc[4];
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[d][v] = 0.0f;
  float m_run = -1e30f, l_run = 0.0f;

  // ds_read_b64_tr_b16 addressing for the V^T operand (see header comment);
  // row v_row (+ 16 u, + 8) keeps v_row & 3, so its 64-byte group d sits at
  // d ^ v_sw
  const int j16 = lane & 15, G = lane >> 4, hh = G >> 1;
  const int v_row = 4 * hh + (j16 >> 2);
  const int v_colb = 2 * (16 * (G & 1) + 4 * (j16 & 3));
  const int v_sw = v_row & 3;

  const int nkb_all = p.causal ? (q0 + BQ + BKV - 1) / BKV : p.S / BKV;
  // a shard's key range is kb_per blocks of 64 keys
  const int kb_begin = p.nsplit > 1 ? split * p.kb_per * (64 / BKV) : 0;
  const int nkb = p.nsplit > 1 ? min(nkb_all, kb_begin + p.kb_per * (64 / BKV)) : nkb_all;   // one past the last block
  const int wave_last_q = q0 + 32 * w + 31;

  if (kb_begin < nkb) gload(kb_begin, 0);
  // Every load so far (the Q fragments included) has landed on every path
  // into the loop; without this the wait insertion cannot tell on the path
  // that skips the first block, and waits on the next block's prefetch
  // before each S^T step.
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  __syncthreads();
  // Two blocks per loop trip, so that each block's stage is a constant and
  // its LDS offset folds into the read instructions.
  auto block = [&](auto stage_c, int kb) {
    constexpr int cur = decltype(stage_c)::value;
    // the other stage was finished with before the last barrier
    if (kb + 1 < nkb) gload(kb + 1, cur ^ 1);
    const int k0 = kb * BKV;
    if (!p.causal || k0 <= wave_last_q) {
      const char* ks = smem + cur * STAGE;
      const char* vs = ks + T_BYTES;
      // S^T = K Q^T for NSUB 32-key sub-tiles: this lane's column holds
      // query qi, keys k0 + 32 t + 8 (v / 4) + 4 h + v % 4 in element v of
      // sub-tile t
      // While it issues the S^T products a wave takes issue priority over the
      // other waves of its SIMD (in their softmax or P V steps), which keeps
      // the matrix pipe fed between their shorter MFMA runs.
      __builtin_amdgcn_s_setprio(1);
      f32x16 sacc[NSUB];
#pragma unroll
      for (int t = 0; t < NSUB; ++t) {
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[t][v] = 0.0f;
        const int r = 32 * t + col;
#pragma unroll
        for (int ds = 0; ds < 8; ++ds) {
          const bf16x8 kf = lds_read_b128(ks + r * RP + (((2 * ds + h) ^ (r & 15)) << 4));
          sacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ds], sacc[t], 0, 0, 0);
        }
      }
      __builtin_amdgcn_s_setprio(0);
      // causal mask on the raw scores; the scale (> 0) is folded into the
      // exponent: p = 2^(s c - m) with m the subtracted maximum in log2 units
      if (p.causal && k0 + BKV - 1 > q0 + 32 * w) {   // wave-uniform: only blocks on the diagonal
#pragma unroll
        for (int t = 0; t < NSUB; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = k0 + 32 * t + 8 * (v >> 2) + 4 * h + (v & 3);
            if (key > qi) sacc[t][v] = -__builtin_inff();
          }
      }
      const float sl2 = p.scale_log2;
      float lsum = 0.0f;
      bf16x8 pf[2 * NSUB];
      auto weights = [&]() {
        lsum = 0.0f;
#pragma unroll
        for (int t = 0; t < NSUB; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[t][v], sl2, -m_run));
            lsum += e;
            pf[2 * t + (v >> 3)][v & 7] = (__bf16)e;
          }
      };
      // Lazy rescaling: m moves only when the block's maximum exceeds it by
      // more than 8 (log2 units), so every p stays <= 2^8 (exact range in
      // fp32 and bf16; the softmax does not depend on the constant
      // subtracted) and O and l are rescaled in few blocks.  The block
      // maximum itself is needed only then: the weights are formed with the
      // current m first, and a lane whose 16 * NSUB weights sum to at most 2^8 has
      // none above 2^8, i.e. no score that would move m.  Only when some
      // lane's sum exceeds 2^8 (or is inf / NaN, as on the first block,
      // where m starts at -1e30) does the wave take the maximum over both
      // halves of each query's keys, move m where the rule says so, and
      // form the weights again; m, the weights and the sums are those of
      // taking the maximum on every block.
      weights();
      if (__builtin_amdgcn_ballot_w64(!(lsum <= 256.0f)) != 0) {
        float mloc = -__builtin_inff();
#pragma unroll
        for (int t = 0; t < NSUB; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v) mloc = fmaxf(mloc, sacc[t][v]);
        // the partner lane (lane ^ 32) holds the other keys of this query
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
        const float m_blk = mloc * sl2;
        const bool move = m_blk > m_run + 8.0f;
        if (__builtin_amdgcn_ballot_w64(move) != 0) {
          const float m_new = move ? m_blk : m_run;
          const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);   // exactly 1 where m_run stays
          l_run *= alpha;
#pragma unroll
          for (int d = 0; d < 4; ++d) oacc[d] *= alpha;
          m_run = m_new;
          weights();
        }
      }
      l_run += lsum;
      // O^T += V^T P^T, BKV / 16 steps of 16 keys
#pragma unroll
      for (int u = 0; u < BKV / 16; ++u) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const char* base = vs + (16 * u + v_row) * RP + 64 * (d ^ v_sw) + v_colb;
          const i16x4 lo = lds_read_tr16(base);
          const i16x4 hi = lds_read_tr16(base + 8 * RP);
          // whole-vector reinterpretation (per-element casts were lowered to
          // reads of the first dword only)
          const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          oacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[u], oacc[d], 0, 0, 0);
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's loads of the next tiles landed
    __syncthreads();
  };
  for (int kb = kb_begin; kb < nkb; kb += 2) {
    block(std::integral_constant<int, 0>{}, kb);
    if (kb + 1 < nkb) block(std::integral_constant<int, 1>{}, kb + 1);
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (p.nsplit > 1) {
    // one shard of the key loop: unnormalised output and (m, l) for the combine
    const int64_t tq = tok0 + qi;
    float* orow = p.Opart + ((int64_t)split * p.B * p.S + tq) * (p.H * DH) + head * DH;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 o = {oacc[d][4 * g + 0], oacc[d][4 * g + 1], oacc[d][4 * g + 2], oacc[d][4 * g + 3]};
        *(f32x4*)(orow + 32 * d + 8 * g + 4 * h) = o;
      }
    if (h == 0) {
      const int64_t st = ((int64_t)split * p.B * p.S + tq) * p.H + head;
      p.Mpart[st] = m_run;
      p.Lpart[st] = l_tot;
    }
    return;
  }
  // ---- normalise and store O[query][head*128 + d] ------------------------------
  if (p.lse && h == 0) p.lse[(tok0 + qi) * p.H + head] = m_run + __builtin_amdgcn_logf(l_tot);
  const float inv = 1.0f / l_tot;
  uint16_t* orow = p.O + (tok0 + qi) * p.ldo + head * DH;
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 o = {(__bf16)(oacc[d][4 * g + 0] * inv), (__bf16)(oacc[d][4 * g + 1] * inv),
                  (__bf16)(oacc[d][4 * g + 2] * inv), (__bf16)(oacc[d][4 * g + 3] * inv)};
      *(bf16x4*)(orow + 32 * d + 8 * g + 4 * h) = o;
    }
}

// One thread per (token, head, 4 of the 128 output columns).  The shards are
// folded in order s = 0..nsplit-1, so the result does not depend on timing.
__global__ __launch_bounds__(256) void attention_combine_kernel(AttnParams p) {
  const int64_t T = (int64_t)p.B * p.S;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= T * p.H * (DH / 4)) return;
  const int c4 = (int)(idx % (DH / 4));
  const int64_t th = idx / (DH / 4);          // token * H + head
  const int64_t t = th / p.H;
  const int head = (int)(th - t * p.H);
  const int64_t sstride = T * p.H;
  // with a causal mask, shard s holds keys for this row only if its first key
  // s * kb_per * 64 is at or before the row's position; the later shards were
  // not written (their share of the sum is zero)
  const int nparts = p.causal ? min(p.nsplit, (int)(t % p.S) / (p.kb_per * 64) + 1) : p.nsplit;
  float M = -3.0e38f;
  for (int s = 0; s < nparts; ++s) M = fmaxf(M, p.Mpart[s * sstride + th]);
  float L = 0.0f;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int s = 0; s < nparts; ++s) {
    const float w = __builtin_amdgcn_exp2f(p.Mpart[s * sstride + th] - M);
    L += w * p.Lpart[s * sstride + th];
    acc += w * *(const f32x4*)(p.Opart + (s * T + t) * (int64_t)(p.H * DH) + head * DH + 4 * c4);
  }
  if (p.lse && c4 == 0) p.lse[th] = M + __builtin_amdgcn_logf(L);
  const float inv = 1.0f / L;
  const bf16x4 o = {(__bf16)(acc[0] * inv), (__bf16)(acc[1] * inv), (__bf16)(acc[2] * inv), (__bf16)(acc[3] * inv)};
  *(bf16x4*)(p.O + t * p.ldo + head * DH + 4 * c4) = o;
}

}  // namespace

hipError_t launch_attention_combine(const AttnParams& p, hipStream_t s) {
  const int64_t n = (int64_t)p.B * p.S * p.H * (DH / 4);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(attention_combine_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnParams& p, hipStream_t s) {
  const unsigned nwg = (unsigned)(p.S / BQ) * p.B * p.H * p.nsplit;
  // CU count per device, looked up once (racing first calls store the same value)
  static int cus[64] = {};
  int dev = 0, ncu = 256;
  if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64) {
    if (cus[dev] == 0) {
      int n = 0;
      if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) cus[dev] = n;
    }
    if (cus[dev] > 0) ncu = cus[dev];
  }
  if (nwg < (unsigned)ncu)
    hipLaunchKernelGGL(attention_kernel<64>, dim3(nwg), dim3(NT), 0, s, p);
  else
    hipLaunchKernelGGL(attention_kernel<32>, dim3(nwg), dim3(NT), 0, s, p);
  return hipGetLastError();
}

}  // namespace partir
