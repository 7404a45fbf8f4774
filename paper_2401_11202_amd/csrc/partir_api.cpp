// libpartir host side: argument validation, the loop-nest planner and launch.
//
// Every entry point follows the same three steps:
//  1. validate the call against PartIR:Core's typing rules (TSlice needs the
//     axis size to divide the sliced dim exactly; TTile / TSum fix the result
//     shapes; one axis may not be nested in itself, Sec. 5.2.3) and against
//     the layout contract of the kernels, returning a status before anything
//     is enqueued;
//  2. plan: enumerate the virtual shards of the nest and turn them into a
//     short list of kernel launches whose grids span all shards at once
//     (slices become base offsets, #tile results offset stores, #sum either a
//     fused accumulator or fp32 partials plus an ordered reduction);
//  3. enqueue the launches on the caller's stream.
// The plan-query entry points run steps 1-2 only and need no GPU.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/partir.h"
#include "kernels.h"

namespace partir {
namespace {

constexpr int kNumCU = 256;           // MI355X compute units: a grid below this underfills
// Tile-order grouping for L2 reuse: consecutive workgroups walk group_m tile
// rows before the next tile column; wide grids want shorter groups.
// Tile-order grouping of the bf16 GEMM: consecutive tiles walk group_m tile
// rows before moving to the next tile column, so the 32 tiles one XCD runs at
// a time form a 4 x 8 block of the output, whose operands are 12 row blocks
// (a 2 x 16 block needs 18): the least L2 -> fabric traffic per k step.
int group_m_for(int /*tiles_n*/) { return 4; }
constexpr size_t kWsAlign = 256;

thread_local std::string g_error;
thread_local std::string g_plan_text;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = std::string(partir_status_string(status)) + ": " + buf;
  return status;
}

size_t align_up(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }
int elem_bytes(int dt) { return dt == PARTIR_BF16 ? 2 : 4; }
bool valid_dtype(int dt) { return dt == PARTIR_F32 || dt == PARTIR_BF16; }

// ---------------------------------------------------------------------------
// Plans
// ---------------------------------------------------------------------------
enum LaunchKind { L_GEMM_BF16, L_GEMM_F32, L_REDUCE, L_ATTN, L_ATTN_COMBINE, L_RMS, L_ACT_BWD, L_COLSUM,
                  L_GEMM_BF16_PARTS, L_ATTN_BWD, L_RMS_PARTS, L_GEMM_BF16_FIXUP, L_GEMM_BF16_PARTS_FIXUP };

struct Launch {
  LaunchKind kind;
  std::string name;
  std::string text;
  GemmParams gemm{};
  GemmF32Params gemm32{};
  ReduceParams reduce{};
  AttnParams attn{};
  RmsParams rms{};
  ActBwdParams act{};
  ColSumParams cs{};
  std::shared_ptr<GemmParts> parts;   // L_GEMM_BF16_PARTS: the device-local arrays
  std::shared_ptr<RmsParts> rms_parts;   // L_RMS_PARTS
  AttnBwdParams attn_bwd{};
};

struct Plan {
  std::vector<Launch> launches;
  int n_shards = 1;
  int n_tile_loops = 0;
  int n_sum_loops = 0;
  int n_sum_splitk = 0;
  size_t ws_bytes = 0;
  double flops = 0;
};

// ---------------------------------------------------------------------------
// Tracing
// ---------------------------------------------------------------------------
struct TraceRec {
  std::string name;
  hipEvent_t start, stop;
};
std::mutex g_trace_mu;
bool g_trace_on = false;
std::vector<TraceRec> g_trace_pending;
std::map<std::string, std::pair<int64_t, double>> g_trace_totals;

// ---------------------------------------------------------------------------
// GEMM planning
// ---------------------------------------------------------------------------
struct GemmSpec {
  // operands (NULL while only planning)
  const void* A = nullptr;
  const void* B[3] = {nullptr, nullptr, nullptr};
  void* C[3] = {nullptr, nullptr, nullptr};
  const float* bias[3] = {nullptr, nullptr, nullptr};
  const float* resid = nullptr;
  int64_t lda = 0, ldb = 0, ldc = 0, ldr = 0;
  int64_t M = 0, N = 0, K = 0;
  int ngroups = 1;
  int ab_dtype = PARTIR_BF16, c_dtype = PARTIR_BF16;
  int b_nk = 1;
  int rm = 1, rn = 1, rk = 1;   // #tile shards on M, N; #sum shards on K
  int act = 0;
  bool resid_add = false;
  int sum_impl = PARTIR_SUM_AUTO;
  void* aux = nullptr;          // bf16 pre-activation output (kept for a backward pass)
  bool tail_ok = false;         // the caller's workspace region holds gemm_ws_bytes (tail split allowed)
  bool a_mn = false;            // bf16 A stored [K, M] (leading dim lda) instead of [M, K]
  const char* name = "gemm";    // role, used as the trace name
  const char* label = "gemm";   // loop nest, for the plan text
};

int64_t gemm_tiles(const GemmSpec& g) {
  const int64_t tile = g.ab_dtype == PARTIR_BF16 ? gemm_bf16_tile_m() : gemm_f32_tile();
  return g.rm * cdiv(g.M / g.rm, tile) * g.ngroups * g.rn * cdiv(g.N / g.rn, tile);
}

bool gemm_uses_splitk(const GemmSpec& g) {
  if (g.rk <= 1) return false;
  if (g.sum_impl == PARTIR_SUM_SPLITK) return true;
  if (g.sum_impl == PARTIR_SUM_FUSED) return false;
  return gemm_tiles(g) < kNumCU;   // too few output tiles: spread the K shards too
}

// Load balance of the last wave: with ntiles = q * kNumCU + r output tiles
// (0 < r <= kNumCU / 2), the r tiles of the partial last wave run as `parts`
// workgroups each over consecutive K ranges, so the last wave holds
// r * parts <= kNumCU shorter workgroups instead of r whole ones; a fixup
// launch adds the parts in ascending K order (deterministic) and runs the
// epilogue.  Returns parts (1: no split) and the first split tile.
int gemm_tail_parts(const GemmSpec& g, int64_t* tail_base) {
  *tail_base = 0;
  if (!g.tail_ok || g.ab_dtype != PARTIR_BF16 || gemm_uses_splitk(g)) return 1;
  const int64_t ntiles = gemm_tiles(g), r = ntiles % kNumCU, nk = cdiv(g.K, 64);
  int parts = 1;
  while (parts < 4 && 2 * parts * r <= kNumCU && nk >= 2 * parts * 8) parts *= 2;   // >= 8 K tiles a part
  if (r == 0 || parts == 1 || (r * parts) % 8) return 1;   // the XCD schedule wants multiples of 8
  *tail_base = ntiles - r;
  return parts;
}

size_t gemm_ws_bytes(const GemmSpec& g) {
  if (gemm_uses_splitk(g)) return align_up((size_t)g.rk * g.M * g.N * sizeof(float));
  int64_t base;
  const int parts = gemm_tail_parts(g, &base);
  return parts > 1 ? align_up((size_t)(gemm_tiles(g) - base) * parts * kGemmTailPartBytes) : 0;
}

std::string describe_gemm(const GemmSpec& g, int64_t grid, bool split) {
  char buf[512];
  snprintf(buf, sizeof buf,
           "%s: C[%lld,%lld]%s = A[%lld,%lld] . B[%lld,%lld]; #tile M x%d (rows %lld/shard), "
           "#tile N x%d (cols %lld/shard)%s; #sum K x%d (%lld/shard) %s; grid %lld WGs",
           g.label, (long long)g.M, (long long)(g.N * g.ngroups), g.ngroups > 1 ? " (groups)" : "",
           (long long)g.M, (long long)g.K, (long long)g.K, (long long)(g.N * g.ngroups), g.rm,
           (long long)(g.M / g.rm), g.rn, (long long)(g.N / g.rn),
           g.ngroups > 1 ? " per group" : "", g.rk, (long long)(g.K / g.rk),
           g.rk <= 1 ? "(none)" : (split ? "split-K fp32 partials + ordered reduce" : "fused in accumulator, r ascending"),
           (long long)grid);
  std::string t = buf;
  if (g.ab_dtype == PARTIR_BF16 && (g.a_mn || !g.b_nk)) {
    t += "; read in place:";
    if (g.a_mn) t += " A as [K, M]";
    if (!g.b_nk) t += " B as [K, N]";
  }
  return t;
}

// Appends the launches of one GEMM to the plan (returns how many).  `ws`
// points at this GEMM's region of gemm_ws_bytes(g) bytes (split-K partials or
// the tail parts).
int plan_gemm(const GemmSpec& g, void* ws, Plan& plan) {
  const bool split = gemm_uses_splitk(g);
  if (g.rk > 1) {
    plan.n_sum_loops += 1;
    if (split) plan.n_sum_splitk += 1;
  }
  const int epi_store = g.resid_add ? EPI_RESID_F32 : (g.c_dtype == PARTIR_BF16 ? EPI_BF16 : EPI_F32);
  Launch L;
  if (g.ab_dtype == PARTIR_BF16) {
    const int tile = gemm_bf16_tile_m();
    GemmParams& p = L.gemm;
    p.A = (const uint16_t*)g.A;
    for (int i = 0; i < 3; ++i) {
      p.B[i] = (const uint16_t*)g.B[i];
      p.C[i] = g.C[i];
      p.bias[i] = split ? nullptr : g.bias[i];
    }
    p.resid = g.resid;
    p.partial = (float*)ws;
    p.aux = g.aux;
    p.lda = g.lda; p.ldb = g.ldb; p.ldc = g.ldc; p.ldr = g.ldr;
    p.part_ld = g.N; p.part_stride = g.M * g.N;
    p.M = (int)g.M; p.N = (int)g.N; p.K = (int)g.K; p.ngroups = g.ngroups;
    p.rm = g.rm; p.ms = (int)(g.M / g.rm); p.tpm = (int)cdiv(p.ms, tile);
    p.rn = g.rn; p.ns = (int)(g.N / g.rn); p.tpn = (int)cdiv(p.ns, tile);
    p.rk = g.rk; p.ks = (int)(g.K / g.rk);
    p.tiles_m = p.rm * p.tpm;
    p.tiles_n = g.ngroups * p.rn * p.tpn;
    p.nsplit = split ? g.rk : 1;
    p.group_m = group_m_for(p.tiles_n);
    p.act = split ? 0 : g.act;
    // a kept pre-activation needs the whole K sum in the tile (never split:
    // only the up-projection, which has no #sum, asks for it)
    p.epi = split ? EPI_PARTIAL : (g.aux ? EPI_BF16_SAVE : epi_store);
    p.a_mn = g.a_mn;
    p.b_mn = !g.b_nk;   // B stored [K, N]
    int64_t tail_base;
    p.tail_parts = gemm_tail_parts(g, &tail_base);
    p.tail_base = (int)tail_base;
    p.tail_kt = (int)cdiv(cdiv(g.K, 64), p.tail_parts);
    p.tail_ws = p.tail_parts > 1 ? (float*)ws : nullptr;
    L.kind = L_GEMM_BF16;
    L.name = g.name;
    const int64_t ntiles = (int64_t)p.tiles_m * p.tiles_n;
    L.text = describe_gemm(g, p.tail_parts > 1 ? tail_base + (ntiles - tail_base) * p.tail_parts : ntiles * p.nsplit,
                           split);
    if (p.tail_parts > 1) {
      char buf[200];
      snprintf(buf, sizeof buf, "; the last %lld tiles as %d K parts of %d K tiles each",
               (long long)(ntiles - tail_base), p.tail_parts, p.tail_kt);
      L.text += buf;
      plan.launches.push_back(L);
      Launch Fx = L;
      Fx.kind = L_GEMM_BF16_FIXUP;
      Fx.name = std::string(g.name) + ".fixup";
      snprintf(buf, sizeof buf, "%s.fixup: %lld tiles = sum of their %d K parts in ascending order, then the epilogue",
               g.name, (long long)(ntiles - tail_base), p.tail_parts);
      Fx.text = buf;
      plan.launches.push_back(Fx);
      return 2;
    }
  } else {
    const int tile = gemm_f32_tile();
    GemmF32Params& p = L.gemm32;
    p.A = (const float*)g.A;
    p.B = (const float*)g.B[0];
    p.C = split ? (float*)ws : (float*)g.C[0];
    p.lda = g.lda; p.ldb = g.ldb;
    p.ldc = split ? g.N : g.ldc;
    p.part_stride = g.M * g.N;
    p.M = (int)g.M; p.N = (int)g.N; p.K = (int)g.K; p.b_nk = g.b_nk;
    p.rm = g.rm; p.ms = (int)(g.M / g.rm); p.tpm = (int)cdiv(p.ms, tile);
    p.rn = g.rn; p.ns = (int)(g.N / g.rn); p.tpn = (int)cdiv(p.ns, tile);
    p.rk = g.rk; p.ks = (int)(g.K / g.rk);
    p.tiles_m = p.rm * p.tpm; p.tiles_n = p.rn * p.tpn;
    p.nsplit = split ? g.rk : 1;
    p.epi = split ? EPI_PARTIAL : EPI_F32;
    L.kind = L_GEMM_F32;
    L.name = g.name;
    L.text = describe_gemm(g, (int64_t)p.tiles_m * p.tiles_n * p.nsplit, split);
  }
  plan.launches.push_back(L);
  if (split) {
    Launch R;
    R.kind = L_REDUCE;
    R.name = std::string(g.name) + ".reduce";
    ReduceParams& r = R.reduce;
    r.partial = (const float*)ws;
    r.part_ld = g.N; r.part_stride = g.M * g.N;
    r.R = g.rk; r.M = (int)g.M; r.N = (int)g.N;
    r.C = g.C[0]; r.ldc = g.ldc;
    r.bias = g.bias[0];
    r.resid = g.resid; r.ldr = g.ldr;
    r.act = g.act;
    r.out_bf16 = (!g.resid_add && g.c_dtype == PARTIR_BF16);
    r.resid_add = g.resid_add;
    char buf[256];
    snprintf(buf, sizeof buf, "splitk_reduce: C[%lld,%lld] = sum_{r=0..%d} partial[r] (in-device all_reduce)%s%s",
             (long long)g.M, (long long)g.N, g.rk - 1, g.bias[0] ? " + bias" : "",
             g.resid_add ? " + residual" : "");
    R.text = buf;
    plan.launches.push_back(R);
    return 2;
  }
  return 1;
}

// ---------------------------------------------------------------------------
// Launch
// ---------------------------------------------------------------------------
hipError_t run_one(const Launch& L, hipStream_t s) {
  switch (L.kind) {
    case L_GEMM_BF16: return launch_gemm_bf16(L.gemm, s);
    case L_GEMM_F32: return launch_gemm_f32(L.gemm32, s);
    case L_REDUCE: return launch_splitk_reduce(L.reduce, s);
    case L_ATTN: return launch_attention(L.attn, s);
    case L_ATTN_COMBINE: return launch_attention_combine(L.attn, s);
    case L_RMS: return launch_rmsnorm(L.rms, s);
    case L_ACT_BWD: return launch_act_backward(L.act, s);
    case L_COLSUM: return launch_colsum(L.cs, s);
    case L_GEMM_BF16_PARTS: return launch_gemm_bf16_parts(L.gemm, *L.parts, s);
    case L_GEMM_BF16_FIXUP: return launch_gemm_bf16_fixup(L.gemm, s);
    case L_GEMM_BF16_PARTS_FIXUP: return launch_gemm_bf16_parts_fixup(L.gemm, *L.parts, s);
    case L_ATTN_BWD: return launch_attention_backward(L.attn_bwd, s);
    case L_RMS_PARTS: return launch_rmsnorm_parts(L.rms, *L.rms_parts, s);
  }
  return hipErrorInvalidValue;
}

void keep_plan_text(const Plan& plan, const char* what) {
  std::string t = std::string(what) + ": " + std::to_string(plan.n_shards) + " virtual shards, " +
                  std::to_string(plan.n_tile_loops) + " #tile loops, " + std::to_string(plan.n_sum_loops) +
                  " #sum loops (" + std::to_string(plan.n_sum_splitk) + " split-K), workspace " +
                  std::to_string(plan.ws_bytes) + " B\n";
  for (size_t i = 0; i < plan.launches.size(); ++i)
    t += "  [" + std::to_string(i) + "] " + plan.launches[i].text + "\n";
  g_plan_text = t;
  const char* dump = getenv("PARTIR_DUMP_PLAN");
  if (dump && dump[0] == '1') fputs(t.c_str(), stderr);
}

int execute(const Plan& plan, void* stream) {
  const char* force = getenv("PARTIR_FAIL_LAUNCH");
  if (force && force[0] == '1') return fail(PARTIR_E_HIP, "launch failure forced by PARTIR_FAIL_LAUNCH");
  hipStream_t s = (hipStream_t)stream;
  (void)hipGetLastError();
  for (const Launch& L : plan.launches) {
    bool traced = false;
    TraceRec rec;
    {
      std::lock_guard<std::mutex> lk(g_trace_mu);
      traced = g_trace_on;
    }
    if (traced) {
      rec.name = L.name;
      if (hipEventCreate(&rec.start) != hipSuccess || hipEventCreate(&rec.stop) != hipSuccess)
        return fail(PARTIR_E_HIP, "hipEventCreate failed");
      if (hipEventRecord(rec.start, s) != hipSuccess) return fail(PARTIR_E_HIP, "hipEventRecord failed");
    }
    const hipError_t e = run_one(L, s);
    if (e != hipSuccess) return fail(PARTIR_E_HIP, "launch of %s failed: %s", L.name.c_str(), hipGetErrorString(e));
    if (traced) {
      if (hipEventRecord(rec.stop, s) != hipSuccess) return fail(PARTIR_E_HIP, "hipEventRecord failed");
      std::lock_guard<std::mutex> lk(g_trace_mu);
      g_trace_pending.push_back(rec);
    }
  }
  return PARTIR_OK;
}

int check_ws(const Plan& plan, void* ws, size_t ws_bytes) {
  if (ws_bytes < plan.ws_bytes)
    return fail(PARTIR_E_WORKSPACE, "workspace of %zu bytes, need %zu", ws_bytes, plan.ws_bytes);
  if (plan.ws_bytes > 0 && ws == nullptr) return fail(PARTIR_E_NULL, "workspace pointer is NULL");
  if (plan.ws_bytes > 0 && !aligned16(ws)) return fail(PARTIR_E_LAYOUT, "workspace not 16-byte aligned");
  return PARTIR_OK;
}

// ---------------------------------------------------------------------------
// partir_loop_matmul
// ---------------------------------------------------------------------------
struct MatmulArgs {
  const void *A = nullptr, *B = nullptr;
  void* C = nullptr;
  int64_t M, N, K, lda, ldb, ldc;
  int ab, c, b_layout, tile_axis, sum_axis, R, sum_impl;
};

constexpr int64_t kBf16MaxLd = (int64_t)1 << 24;

int validate_matmul(const MatmulArgs& a, bool with_ptrs) {
  // Empty operands are legal: a zero-size dim slices into R empty shards
  // (n_d = 0 satisfies TSlice), and a #sum over K = 0 is the empty sum.
  if (a.M < 0 || a.N < 0 || a.K < 0) return fail(PARTIR_E_SHAPE, "M, N, K must be >= 0");
  if (with_ptrs && ((a.M * a.K > 0 && !a.A) || (a.K * a.N > 0 && !a.B) || (a.M * a.N > 0 && !a.C)))
    return fail(PARTIR_E_NULL, "A, B and C must be non-NULL (unless empty)");
  if (a.M > (1 << 30) || a.N > (1 << 30) || a.K > (1 << 30)) return fail(PARTIR_E_SHAPE, "dims above 2^30");
  if (a.R < 1) return fail(PARTIR_E_UNSUPPORTED, "R = %d: a loop needs at least one shard", a.R);
  if (a.tile_axis != PARTIR_AXIS_NONE && a.tile_axis != PARTIR_AXIS_M && a.tile_axis != PARTIR_AXIS_N) {
    if (a.tile_axis == PARTIR_AXIS_K)
      return fail(PARTIR_E_AXIS, "#tile over K: K is contracted, so its shards must be summed, not concatenated");
    return fail(PARTIR_E_AXIS, "tile_axis %d is not NONE, M or N", a.tile_axis);
  }
  if (a.sum_axis != PARTIR_AXIS_NONE && a.sum_axis != PARTIR_AXIS_K) {
    if (a.sum_axis == a.tile_axis)
      return fail(PARTIR_E_AXIS, "axis %d is both tiled and summed", a.sum_axis);
    return fail(PARTIR_E_AXIS, "sum_axis %d: only the contracted dim K can carry #sum", a.sum_axis);
  }
  if (!valid_dtype(a.ab) || !valid_dtype(a.c)) return fail(PARTIR_E_DTYPE, "dtype must be F32 or BF16");
  if (a.ab == PARTIR_F32 && a.c != PARTIR_F32) return fail(PARTIR_E_DTYPE, "f32 inputs need an f32 output");
  if (a.b_layout != PARTIR_B_KN && a.b_layout != PARTIR_B_NK) return fail(PARTIR_E_LAYOUT, "b_layout %d", a.b_layout);
  if (a.sum_impl < PARTIR_SUM_AUTO || a.sum_impl > PARTIR_SUM_SPLITK)
    return fail(PARTIR_E_UNSUPPORTED, "sum_impl %d", a.sum_impl);
  if (a.tile_axis == PARTIR_AXIS_M && a.M % a.R) return fail(PARTIR_E_DIVISIBILITY, "R=%d does not divide M=%lld", a.R, (long long)a.M);
  if (a.tile_axis == PARTIR_AXIS_N && a.N % a.R) return fail(PARTIR_E_DIVISIBILITY, "R=%d does not divide N=%lld", a.R, (long long)a.N);
  if (a.sum_axis == PARTIR_AXIS_K && a.K % a.R) return fail(PARTIR_E_DIVISIBILITY, "R=%d does not divide K=%lld", a.R, (long long)a.K);
  const int eb = elem_bytes(a.ab), vec = 16 / eb;
  const int64_t ldb_min = a.b_layout == PARTIR_B_KN ? a.N : a.K;
  // leading dims matter only for operands that hold elements
  const bool a_used = a.M * a.K > 0, b_used = a.K * a.N > 0, c_used = a.M * a.N > 0;
  if ((a_used && a.lda < a.K) || (b_used && a.ldb < ldb_min) || (c_used && a.ldc < a.N))
    return fail(PARTIR_E_LAYOUT, "leading dim smaller than the row length");
  if ((a_used && a.lda % vec) || (b_used && a.ldb % vec) || (c_used && a.ldc % (16 / elem_bytes(a.c))))
    return fail(PARTIR_E_LAYOUT, "leading dims must keep rows 16-byte aligned");
  if (a.K % vec) return fail(PARTIR_E_LAYOUT, "K must be a multiple of %d", vec);
  if (a.N % 4) return fail(PARTIR_E_LAYOUT, "N must be a multiple of 4");
  const int rk = a.sum_axis == PARTIR_AXIS_K ? a.R : 1;
  const int rn = a.tile_axis == PARTIR_AXIS_N ? a.R : 1;
  if ((a.K / rk) % vec) return fail(PARTIR_E_LAYOUT, "K/R must be a multiple of %d (16-byte shard views)", vec);
  // The bf16 kernel addresses each 64-row block of an operand (64 K rows of
  // an MN-major one) through a buffer descriptor whose byte range is a 32-bit
  // number, and masks a lane with offset bit 31: 128 * ld bytes must stay
  // within 2^31.
  if (a.ab == PARTIR_BF16 && ((a_used && a.lda > kBf16MaxLd) || (b_used && a.ldb > kBf16MaxLd)))
    return fail(PARTIR_E_SHAPE, "bf16 operands: leading dims above 2^24 elements are not addressable");
  // output tiles (64 x 64 at the smallest, never straddling a shard) times
  // K shards index the grid in 32 bits
  const int64_t rm = a.tile_axis == PARTIR_AXIS_M ? a.R : 1;
  if (c_used && rm * cdiv(a.M / rm, 64) * rn * cdiv(a.N / rn, 64) * (int64_t)rk > ((int64_t)1 << 31) - 1)
    return fail(PARTIR_E_SHAPE, "C[%lld,%lld] with R=%d has more output tiles than a launch can index",
                (long long)a.M, (long long)a.N, a.R);
  if ((a.N / rn) % 4) return fail(PARTIR_E_LAYOUT, "N/R must be a multiple of 4 (16-byte shard views)");
  if (a.ab == PARTIR_BF16 && a.b_layout == PARTIR_B_KN && ((a.N % 8) || ((a.N / rn) % 8)))
    return fail(PARTIR_E_LAYOUT, "bf16 B as [K, N]: N and N/R must be multiples of 8 (16-byte rows of B)");
  if (with_ptrs && (!aligned16(a.A) || !aligned16(a.B) || !aligned16(a.C)))
    return fail(PARTIR_E_LAYOUT, "A, B and C must be 16-byte aligned");
  return PARTIR_OK;
}

// C[M, N] = epilogue(0): the #sum over an empty contraction (K = 0), done by
// the ordered reduction with no partials.
void plan_empty_sum(void* C, int64_t M, int64_t N, int64_t ldc, bool out_bf16, const float* bias,
                    const float* resid, int64_t ldr, bool resid_add, const char* name, Plan& plan) {
  Launch R;
  R.kind = L_REDUCE;
  R.name = name;
  ReduceParams& r = R.reduce;
  r.partial = nullptr; r.part_ld = 0; r.part_stride = 0;
  r.R = 0; r.M = (int)M; r.N = (int)N;
  r.C = C; r.ldc = ldc; r.bias = bias; r.resid = resid; r.ldr = ldr;
  r.act = 0; r.out_bf16 = out_bf16; r.resid_add = resid_add;
  char buf[200];
  snprintf(buf, sizeof buf, "empty_sum: C[%lld,%lld] = sum over K = 0 (zero)%s", (long long)M, (long long)N,
           bias ? " + bias" : "");
  R.text = buf;
  plan.launches.push_back(R);
}

GemmSpec matmul_spec(const MatmulArgs& a) {
  GemmSpec g;
  g.A = a.A; g.B[0] = a.B; g.C[0] = a.C;
  g.lda = a.lda; g.ldb = a.ldb; g.ldc = a.ldc;
  g.M = a.M; g.N = a.N; g.K = a.K;
  g.ab_dtype = a.ab; g.c_dtype = a.c; g.b_nk = a.b_layout == PARTIR_B_NK;
  g.rm = a.tile_axis == PARTIR_AXIS_M ? a.R : 1;
  g.rn = a.tile_axis == PARTIR_AXIS_N ? a.R : 1;
  g.rk = a.sum_axis == PARTIR_AXIS_K ? a.R : 1;
  g.sum_impl = a.sum_impl;
  g.tail_ok = true;
  g.name = a.ab == PARTIR_BF16 ? "loop_matmul.bf16" : "loop_matmul.f32";
  g.label = "loop_matmul";
  return g;
}

void plan_matmul(const MatmulArgs& a, void* ws, Plan& plan) {
  GemmSpec g = matmul_spec(a);
  plan.ws_bytes = gemm_ws_bytes(g);
  plan.n_shards = g.rm * g.rn * g.rk;
  plan.n_tile_loops = a.tile_axis != PARTIR_AXIS_NONE;
  plan.flops = 2.0 * a.M * a.N * a.K;
  if (a.M == 0 || a.N == 0) return;                 // empty output: nothing to launch
  if (a.K == 0) {
    plan.ws_bytes = 0;
    if (g.rk > 1) plan.n_sum_loops = 1;
    plan_empty_sum(a.C, a.M, a.N, a.ldc, a.c == PARTIR_BF16, nullptr, nullptr, 0, false,
                   a.ab == PARTIR_BF16 ? "loop_matmul.bf16" : "loop_matmul.f32", plan);
    return;
  }
  plan_gemm(g, ws, plan);
}

// ---------------------------------------------------------------------------
// partir_mlp_block
// ---------------------------------------------------------------------------
struct MlpArgs {
  const void *X = nullptr, *W1 = nullptr, *b1 = nullptr, *W2 = nullptr, *b2 = nullptr;
  void* Y = nullptr;
  int64_t T, D, F;
  int in, out, act, Rb, Rm;
  void* Z = nullptr;   // partir_mlp_block_train: the kept pre-activation [T, F] bf16
};

int validate_mlp(const MlpArgs& a, bool with_ptrs) {
  if (a.T < 0 || a.D < 0 || a.F < 0) return fail(PARTIR_E_SHAPE, "T, D, F must be >= 0");
  // an operand must be present only if it will be read (or written)
  if (with_ptrs && ((a.T * a.D > 0 && a.F > 0 && !a.X) || (a.T * a.D * a.F > 0 && (!a.W1 || !a.W2)) ||
                    (a.T * a.D > 0 && !a.Y)))
    return fail(PARTIR_E_NULL, "X, W1, W2 and Y must be non-NULL (unless empty)");
  if (a.T > (1 << 30) || a.D > (1 << 20) || a.F > (1 << 22)) return fail(PARTIR_E_SHAPE, "dims too large");
  if (a.Rb < 1 || a.Rm < 1) return fail(PARTIR_E_UNSUPPORTED, "R_batch and R_model must be >= 1");
  if (a.in != PARTIR_BF16) return fail(PARTIR_E_DTYPE, "in_dtype must be BF16");
  if (!valid_dtype(a.out)) return fail(PARTIR_E_DTYPE, "out_dtype must be F32 or BF16");
  if (a.act != PARTIR_ACT_NONE && a.act != PARTIR_ACT_GELU_ERF) return fail(PARTIR_E_UNSUPPORTED, "act %d", a.act);
  if (a.T % a.Rb) return fail(PARTIR_E_DIVISIBILITY, "R_batch=%d does not divide T=%lld", a.Rb, (long long)a.T);
  if (a.F % a.Rm) return fail(PARTIR_E_DIVISIBILITY, "R_model=%d does not divide F=%lld", a.Rm, (long long)a.F);
  if (a.D % 8 || (a.F / a.Rm) % 8) return fail(PARTIR_E_LAYOUT, "D and F/R_model must be multiples of 8");
  if (with_ptrs && (!aligned16(a.X) || !aligned16(a.W1) || !aligned16(a.W2) || !aligned16(a.Y) ||
                    !aligned16(a.b1) || !aligned16(a.b2) || !aligned16(a.Z)))
    return fail(PARTIR_E_LAYOUT, "tensors must be 16-byte aligned");
  return PARTIR_OK;
}

void plan_mlp(const MlpArgs& a, void* ws, Plan& plan) {
  const size_t h_bytes = align_up((size_t)a.T * a.F * 2);
  char* base = (char*)ws;
  void* H = base;
  // W1 [D, F] and W2 [F, D] are the products' [K, N] right operands, read in place
  GemmSpec g1;
  g1.A = a.X; g1.B[0] = a.W1; g1.b_nk = 0; g1.C[0] = H; g1.bias[0] = (const float*)a.b1;
  g1.lda = a.D; g1.ldb = a.F; g1.ldc = a.F;
  g1.M = a.T; g1.N = a.F; g1.K = a.D;
  g1.c_dtype = PARTIR_BF16; g1.rm = a.Rb; g1.rn = a.Rm; g1.act = a.act; g1.aux = a.Z;
  g1.name = "mlp.up";
  g1.label = "mlp.up   H = act(slice 0 X[b] . slice 1 W1[m])";
  GemmSpec g2;
  g2.A = H; g2.B[0] = a.W2; g2.b_nk = 0; g2.C[0] = a.Y; g2.bias[0] = (const float*)a.b2;
  g2.lda = a.F; g2.ldb = a.D; g2.ldc = a.D;
  g2.M = a.T; g2.N = a.D; g2.K = a.F;
  g2.c_dtype = a.out; g2.rm = a.Rb; g2.rk = a.Rm;
  g2.name = "mlp.down";
  g2.label = "mlp.down Y = sum_m H[:, m] . slice 0 W2[m]";
  plan.ws_bytes = h_bytes + gemm_ws_bytes(g2);
  plan.n_shards = a.Rb * a.Rm;
  plan.n_tile_loops = (a.Rb > 1) + 1;
  plan.flops = 4.0 * a.T * a.D * a.F;
  if (a.T == 0 || a.D == 0) { plan.ws_bytes = 0; return; }   // Y is empty
  if (a.F == 0) {                                              // every model shard is empty: Y = b2
    plan.ws_bytes = 0;
    plan.n_sum_loops = 1;
    plan_empty_sum(a.Y, a.T, a.D, a.D, a.out == PARTIR_BF16, (const float*)a.b2, nullptr, 0, false, "mlp.down", plan);
    return;
  }
  plan_gemm(g1, nullptr, plan);
  plan_gemm(g2, ws ? base + h_bytes : nullptr, plan);
}

// ---------------------------------------------------------------------------
// attention block and decoder layer
// ---------------------------------------------------------------------------
struct AttnArgs {
  const void *X = nullptr, *Wq = nullptr, *Wk = nullptr, *Wv = nullptr, *Wo = nullptr;
  void* Y = nullptr;
  int64_t B, S, D, H, dh;
  int causal;
  float scale;
  int in, out, Rb, Rm;
  void* saved = nullptr;   // partir_attn_block_train: Q | K | V | O | lse kept for the backward
};

int validate_attn_shapes(int64_t B, int64_t S, int64_t D, int64_t H, int64_t dh, int Rb, int Rm) {
  if (B < 0 || S < 0) return fail(PARTIR_E_SHAPE, "B and S must be >= 0 (zero: no tokens, nothing to do)");
  if (D < 1 || H < 1 || dh < 1) return fail(PARTIR_E_SHAPE, "D, n_heads and d_head must be >= 1");
  if (B * S > (1 << 28) || D > (1 << 20)) return fail(PARTIR_E_SHAPE, "sizes too large");
  if (H * dh != D) return fail(PARTIR_E_SHAPE, "n_heads*d_head = %lld != D = %lld", (long long)(H * dh), (long long)D);
  if (dh != 128) return fail(PARTIR_E_SHAPE, "d_head must be 128 (got %lld)", (long long)dh);
  if (S % 128) return fail(PARTIR_E_SHAPE, "S must be a multiple of 128 (got %lld)", (long long)S);
  // the attention kernels address one sequence's rows of Q, K, V by 32-bit byte offsets
  if (S * D * 2 > ((int64_t)1 << 32) - 1)
    return fail(PARTIR_E_SHAPE, "one sequence of S=%lld rows of D=%lld bf16 exceeds 4 GiB", (long long)S, (long long)D);
  if (Rb < 1 || Rm < 1) return fail(PARTIR_E_UNSUPPORTED, "R_batch and R_model must be >= 1");
  if (B % Rb) return fail(PARTIR_E_DIVISIBILITY, "R_batch=%d does not divide B=%lld (batch shards hold whole sequences)", Rb, (long long)B);
  if (H % Rm) return fail(PARTIR_E_DIVISIBILITY, "R_model=%d does not divide n_heads=%lld", Rm, (long long)H);
  return PARTIR_OK;
}

int validate_attn(const AttnArgs& a, bool with_ptrs) {
  int st = validate_attn_shapes(a.B, a.S, a.D, a.H, a.dh, a.Rb, a.Rm);
  if (st) return st;
  const bool empty = a.B * a.S == 0;
  if (with_ptrs && !empty && (!a.X || !a.Wq || !a.Wk || !a.Wv || !a.Wo || !a.Y))
    return fail(PARTIR_E_NULL, "X, W* and Y must be non-NULL");
  if (a.in != PARTIR_BF16) return fail(PARTIR_E_DTYPE, "in_dtype must be BF16");
  if (!valid_dtype(a.out)) return fail(PARTIR_E_DTYPE, "out_dtype must be F32 or BF16");
  if (with_ptrs && (!aligned16(a.X) || !aligned16(a.Wq) || !aligned16(a.Wk) || !aligned16(a.Wv) ||
                    !aligned16(a.Wo) || !aligned16(a.Y)))
    return fail(PARTIR_E_LAYOUT, "tensors must be 16-byte aligned");
  return PARTIR_OK;
}

void plan_attention_launch(char* qkvo, int64_t B, int64_t S, int64_t D, int64_t H, int64_t dh, int causal,
                           float scale, int Rm, Plan& plan, float* lse);

// The QKV projection into (Q, K, V) at qkvo: one launch, three groups.
GemmSpec qkv_spec(const void* Xn, const void* Wq, const void* Wk, const void* Wv, char* qkvo, int64_t T,
                  int64_t D, int Rb, int Rm) {
  const size_t one = align_up((size_t)T * D * 2);
  GemmSpec g;
  g.A = Xn; g.B[0] = Wq; g.B[1] = Wk; g.B[2] = Wv; g.b_nk = 0;   // W{q,k,v} [D, D] as [K, N]
  g.C[0] = qkvo; g.C[1] = qkvo ? qkvo + one : nullptr; g.C[2] = qkvo ? qkvo + 2 * one : nullptr;
  g.ngroups = 3;
  g.lda = D; g.ldb = D; g.ldc = D;
  g.M = T; g.N = D; g.K = D;
  g.c_dtype = PARTIR_BF16; g.rm = Rb; g.rn = Rm;
  g.name = "attn.qkv";
  g.label = "attn.qkv Q|K|V = slice 0 X[b] . slice 1 W{q,k,v}[m]";
  return g;
}

// QKV projection + attention core into (Q, K, V, O) inside the workspace.
// With `gemm_ws` (gemm_ws_bytes of the tail-split qkv_spec) the projection
// may split its last wave.
void plan_attention_core(const void* Xn, const void* Wq, const void* Wk, const void* Wv, char* qkvo,
                         int64_t B, int64_t S, int64_t D, int64_t H, int64_t dh, int causal, float scale,
                         int Rb, int Rm, Plan& plan, float* lse = nullptr, bool tail = false,
                         char* gemm_ws = nullptr) {
  GemmSpec g = qkv_spec(Xn, Wq, Wk, Wv, qkvo, B * S, D, Rb, Rm);
  g.tail_ok = tail;
  plan_gemm(g, gemm_ws, plan);
  plan_attention_launch(qkvo, B, S, D, H, dh, causal, scale, Rm, plan, lse);
}

// The attention core over (Q, K, V) -> O at qkvo (four [T, D] blocks).
void plan_attention_launch(char* qkvo, int64_t B, int64_t S, int64_t D, int64_t H, int64_t dh, int causal,
                           float scale, int Rm, Plan& plan, float* lse) {
  const int64_t T = B * S;
  const size_t one = align_up((size_t)T * D * 2);
  void* Q = qkvo ? qkvo : nullptr;
  void* K = qkvo ? qkvo + one : nullptr;
  void* V = qkvo ? qkvo + 2 * one : nullptr;
  void* O = qkvo ? qkvo + 3 * one : nullptr;
  Launch L;
  L.kind = L_ATTN;
  L.name = "attn.core";
  AttnParams& p = L.attn;
  p.Q = (const uint16_t*)Q; p.K = (const uint16_t*)K; p.V = (const uint16_t*)V; p.O = (uint16_t*)O;
  p.ldq = p.ldk = p.ldv = p.ldo = D;
  p.B = (int)B; p.S = (int)S; p.H = (int)H; p.causal = causal;
  const float sc = scale > 0 ? scale : 1.0f / std::sqrt((float)dh);
  p.scale_log2 = sc * 1.4426950408889634f;
  p.lse = lse;
  char buf[256];
  snprintf(buf, sizeof buf, "attention: loop h [#tile<1>](%lld heads/shard) over %lld sequences x %lld heads, "
           "S=%lld, %s, %lld WGs", (long long)(H / Rm), (long long)B, (long long)H, (long long)S,
           causal ? "causal" : "full", (long long)(S / 128 * B * H));
  L.text = buf;
  plan.launches.push_back(L);
}

size_t attn_core_bytes(int64_t T, int64_t D) { return 4 * align_up((size_t)T * D * 2); }

void plan_attn(const AttnArgs& a, void* ws, Plan& plan) {
  const int64_t T = a.B * a.S;
  if (T == 0) {                                      // no tokens: nothing to do
    plan.n_shards = a.Rb * a.Rm;
    plan.n_tile_loops = (a.Rb > 1) + 1;
    return;
  }
  char* base = (char*)ws;
  // training: Q, K, V, O and the lse go to the caller's buffer, not the workspace
  const size_t core = a.saved ? 0 : attn_core_bytes(T, a.D);
  char* qkvo = a.saved ? (char*)a.saved : base;
  float* lse = a.saved ? (float*)((char*)a.saved + attn_core_bytes(T, a.D)) : nullptr;
  plan_attention_core(a.X, a.Wq, a.Wk, a.Wv, qkvo, a.B, a.S, a.D, a.H, a.dh, a.causal, a.scale, a.Rb, a.Rm, plan,
                      lse);
  GemmSpec g;
  g.A = qkvo ? qkvo + 3 * align_up((size_t)T * a.D * 2) : nullptr;
  g.B[0] = a.Wo; g.b_nk = 0; g.C[0] = a.Y;
  g.lda = a.D; g.ldb = a.D; g.ldc = a.D;
  g.M = T; g.N = a.D; g.K = a.D;
  g.c_dtype = a.out; g.rm = a.Rb; g.rk = a.Rm;
  g.name = "attn.out";
  g.label = "attn.out Y = sum_m O[:, m heads] . slice 0 Wo[m]";
  plan.ws_bytes = core + gemm_ws_bytes(g);
  plan.n_shards = a.Rb * a.Rm;
  plan.n_tile_loops = (a.Rb > 1) + 1;
  const double pairs = a.causal ? (double)a.S * (a.S + 1) / 2 : (double)a.S * a.S;
  plan.flops = 8.0 * T * a.D * a.D + 4.0 * a.B * a.H * pairs * a.dh;
  plan_gemm(g, base ? base + core : nullptr, plan);
}

struct DecArgs {
  void* x = nullptr;
  const void *g1 = nullptr, *g2 = nullptr, *Wq = nullptr, *Wk = nullptr, *Wv = nullptr, *Wo = nullptr,
             *W1 = nullptr, *W2 = nullptr;
  float eps;
  int64_t B, S, D, H, dh, F;
  int Rb, Rm;
};

int validate_dec(const DecArgs& a, bool with_ptrs) {
  int st = validate_attn_shapes(a.B, a.S, a.D, a.H, a.dh, a.Rb, a.Rm);
  if (st) return st;
  if (a.F < 0 || a.F > (1 << 22)) return fail(PARTIR_E_SHAPE, "F out of range");
  const bool empty = a.B * a.S == 0;
  if (with_ptrs && !empty && (!a.x || !a.g1 || !a.Wq || !a.Wk || !a.Wv || !a.Wo ||
                              (a.F > 0 && (!a.g2 || !a.W1 || !a.W2))))
    return fail(PARTIR_E_NULL, "all tensors must be non-NULL");
  if (a.F % a.Rm) return fail(PARTIR_E_DIVISIBILITY, "R_model=%d does not divide F=%lld", a.Rm, (long long)a.F);
  if ((a.F / a.Rm) % 8) return fail(PARTIR_E_LAYOUT, "F/R_model must be a multiple of 8");
  if (!(a.eps >= 0.0f)) return fail(PARTIR_E_SHAPE, "eps must be >= 0");
  if (with_ptrs && (!aligned16(a.x) || !aligned16(a.g1) || !aligned16(a.g2) || !aligned16(a.Wq) ||
                    !aligned16(a.Wk) || !aligned16(a.Wv) || !aligned16(a.Wo) || !aligned16(a.W1) || !aligned16(a.W2)))
    return fail(PARTIR_E_LAYOUT, "tensors must be 16-byte aligned");
  return PARTIR_OK;
}

void plan_rmsnorm(const float* x, const float* g, void* y, int64_t rows, int64_t D, float eps, int Rb, Plan& plan) {
  Launch L;
  L.kind = L_RMS;
  L.name = "rmsnorm";
  RmsParams& p = L.rms;
  p.x = x; p.g = g; p.y = (uint16_t*)y; p.ldx = D; p.ldy = D; p.rows = (int)rows; p.D = (int)D; p.eps = eps;
  char buf[160];
  snprintf(buf, sizeof buf, "rmsnorm: %lld rows x %lld (replicated across model shards, %d batch shards)",
           (long long)rows, (long long)D, Rb);
  L.text = buf;
  plan.launches.push_back(L);
}

void plan_dec(const DecArgs& a, void* ws, Plan& plan) {
  const int64_t T = a.B * a.S;
  if (T == 0) {                                      // no tokens: nothing to do
    plan.n_shards = a.Rb * a.Rm;
    plan.n_tile_loops = (a.Rb > 1) + 2;
    return;
  }
  char* base = (char*)ws;
  const size_t xn_bytes = align_up((size_t)T * a.D * 2);
  const size_t core = attn_core_bytes(T, a.D);
  const size_t h_bytes = align_up((size_t)T * a.F * 2);
  char* xn = base;
  char* qkvo = base ? base + xn_bytes : nullptr;
  char* Hf = base ? base + xn_bytes + core : nullptr;
  char* part = base ? base + xn_bytes + core + h_bytes : nullptr;   // split-K / tail parts, one GEMM at a time
  GemmSpec gq = qkv_spec(xn, a.Wq, a.Wk, a.Wv, qkvo, T, a.D, a.Rb, a.Rm);
  gq.tail_ok = true;

  plan_rmsnorm((const float*)a.x, (const float*)a.g1, xn, T, a.D, a.eps, a.Rb, plan);
  plan_attention_core(xn, a.Wq, a.Wk, a.Wv, qkvo, a.B, a.S, a.D, a.H, a.dh, 1, 0.0f, a.Rb, a.Rm, plan, nullptr,
                      true, part);
  GemmSpec go;
  go.A = qkvo ? qkvo + 3 * align_up((size_t)T * a.D * 2) : nullptr;
  go.B[0] = a.Wo; go.b_nk = 0; go.C[0] = a.x; go.resid = (const float*)a.x; go.resid_add = true;
  go.lda = a.D; go.ldb = a.D; go.ldc = a.D; go.ldr = a.D;
  go.M = T; go.N = a.D; go.K = a.D;
  go.c_dtype = PARTIR_F32; go.rm = a.Rb; go.rk = a.Rm; go.tail_ok = true;
  go.name = "attn.out";
  go.label = "dec.attn_out x += sum_m O[:, m heads] . slice 0 Wo[m]";
  plan_gemm(go, part, plan);
  plan.ws_bytes = xn_bytes + core + std::max(gemm_ws_bytes(gq), gemm_ws_bytes(go));
  plan.n_shards = a.Rb * a.Rm;
  plan.n_tile_loops = (a.Rb > 1) + 2;
  plan.flops = 8.0 * T * a.D * a.D + 4.0 * a.B * a.H * ((double)a.S * (a.S + 1) / 2) * a.dh + 4.0 * T * a.D * a.F;
  if (a.F == 0) return;       // an FFN of width 0 adds the empty sum: x is unchanged
  plan_rmsnorm((const float*)a.x, (const float*)a.g2, xn, T, a.D, a.eps, a.Rb, plan);
  GemmSpec g1;
  g1.A = xn; g1.B[0] = a.W1; g1.b_nk = 0; g1.C[0] = Hf;
  g1.lda = a.D; g1.ldb = a.F; g1.ldc = a.F;
  g1.M = T; g1.N = a.F; g1.K = a.D;
  g1.c_dtype = PARTIR_BF16; g1.rm = a.Rb; g1.rn = a.Rm; g1.act = 1;
  g1.name = "mlp.up";
  g1.label = "dec.ffn_up H = gelu(slice 0 xn[b] . slice 1 W1[m])";
  plan_gemm(g1, nullptr, plan);
  GemmSpec g2;
  g2.A = Hf; g2.B[0] = a.W2; g2.b_nk = 0; g2.C[0] = a.x; g2.resid = (const float*)a.x; g2.resid_add = true;
  g2.lda = a.F; g2.ldb = a.D; g2.ldc = a.D; g2.ldr = a.D;
  g2.M = T; g2.N = a.D; g2.K = a.F;
  g2.c_dtype = PARTIR_F32; g2.rm = a.Rb; g2.rk = a.Rm; g2.tail_ok = true;
  g2.name = "mlp.down";
  g2.label = "dec.ffn_down x += sum_m H[:, m] . slice 0 W2[m]";
  plan_gemm(g2, part, plan);
  plan.ws_bytes = xn_bytes + core + h_bytes +
                  std::max({gemm_ws_bytes(gq), gemm_ws_bytes(go), gemm_ws_bytes(g1), gemm_ws_bytes(g2)});
  plan.n_shards = a.Rb * a.Rm;
  plan.n_tile_loops = (a.Rb > 1) + 2;
  plan.flops = 8.0 * T * a.D * a.D + 4.0 * a.B * a.H * ((double)a.S * (a.S + 1) / 2) * a.dh + 4.0 * T * a.D * a.F;
}

// ---------------------------------------------------------------------------
// partir_attention: the attention core alone, the key axis as a loop
// ---------------------------------------------------------------------------
struct AttnCoreArgs {
  const void *Q = nullptr, *K = nullptr, *V = nullptr;
  void* O = nullptr;
  int64_t B, S, H, dh;
  int causal;
  float scale;
  int Rkv;
  float* lse = nullptr;   // partir_attention_train: per-row base-2 log-sum-exp
};

int validate_attn_core(const AttnCoreArgs& a, bool with_ptrs) {
  int st = validate_attn_shapes(a.B, a.S, a.H * a.dh, a.H, a.dh, 1, 1);
  if (st) return st;
  if (a.Rkv < 1) return fail(PARTIR_E_UNSUPPORTED, "R_kv = %d: a loop needs at least one shard", a.Rkv);
  if ((a.S / 64) % a.Rkv)
    return fail(PARTIR_E_DIVISIBILITY, "R_kv=%d does not divide the %lld key blocks of 64 (S=%lld)", a.Rkv,
                (long long)(a.S / 64), (long long)a.S);
  // one workgroup per (128-query block, sequence, head, part), up to 4 parts a shard
  if ((a.S / 128) * a.B * a.H * a.Rkv > ((int64_t)1 << 29))
    return fail(PARTIR_E_SHAPE, "R_kv=%d gives more than 2^29 (query block, head, shard) workgroups", a.Rkv);
  if (with_ptrs && a.B * a.S > 0 && (!a.Q || !a.K || !a.V || !a.O))
    return fail(PARTIR_E_NULL, "Q, K, V and O must be non-NULL");
  if (with_ptrs && (!aligned16(a.Q) || !aligned16(a.K) || !aligned16(a.V) || !aligned16(a.O)))
    return fail(PARTIR_E_LAYOUT, "Q, K, V and O must be 16-byte aligned");
  return PARTIR_OK;
}

// Parts per key shard of the causal attention core.  A query block needs the
// key blocks up to its own, so under a causal mask the (query block, shard)
// workgroups range from empty to a whole shard; when the grid alone does not
// fill the chip several times over (256 CUs, two attention workgroups each),
// the longest workgroup sets the time.  Each shard of at least 2 x 16 key
// blocks then runs as 2 (or 4) ordered parts of at least 16 blocks, folded in
// key order by the combine like the shards themselves: the same #sum, in
// smaller pieces.  The combine reads, for each row, only the parts whose
// first key is at or before it.
int attn_core_parts(int64_t B, int64_t S, int64_t H, int causal, int Rkv) {
  constexpr int64_t kFillWorkgroups = 4 * 256 * 2;
  constexpr int64_t kMinPartBlocks = 16;
  if (!causal || Rkv < 2) return 1;
  const int64_t kbs = S / 64 / Rkv, wgs = (S / 128) * B * H * Rkv;
  int parts = 1;
  while (parts < 4 && wgs * parts < kFillWorkgroups && kbs % (2 * parts) == 0 && kbs / (2 * parts) >= kMinPartBlocks)
    parts *= 2;
  return parts;
}

void plan_attn_core(const AttnCoreArgs& a, void* ws, Plan& plan) {
  const int64_t T = a.B * a.S, D = a.H * a.dh;
  plan.n_shards = a.Rkv;
  plan.n_tile_loops = 1;                 // the heads loop
  const double pairs = a.causal ? (double)a.S * (a.S + 1) / 2 : (double)a.S * a.S;
  plan.flops = 4.0 * a.B * a.H * pairs * a.dh;
  if (T == 0) return;
  const int parts = attn_core_parts(a.B, a.S, a.H, a.causal, a.Rkv);
  const int nsplit = a.Rkv * parts;
  const size_t o_bytes = align_up((size_t)nsplit * T * D * 4), ml_bytes = align_up((size_t)nsplit * T * a.H * 4);
  if (a.Rkv > 1) {
    plan.ws_bytes = o_bytes + 2 * ml_bytes;
    plan.n_sum_loops = 1;
    plan.n_sum_splitk = 1;
  }
  Launch L;
  L.kind = L_ATTN;
  L.name = "attn.core";
  AttnParams& p = L.attn;
  p.Q = (const uint16_t*)a.Q; p.K = (const uint16_t*)a.K; p.V = (const uint16_t*)a.V; p.O = (uint16_t*)a.O;
  p.ldq = p.ldk = p.ldv = p.ldo = D;
  p.B = (int)a.B; p.S = (int)a.S; p.H = (int)a.H; p.causal = a.causal;
  const float sc = a.scale > 0 ? a.scale : 1.0f / std::sqrt((float)a.dh);
  p.scale_log2 = sc * 1.4426950408889634f;
  p.nsplit = nsplit;
  p.kb_per = (int)(a.S / 64 / nsplit);
  char* base = (char*)ws;
  p.Opart = base ? (float*)base : nullptr;
  p.Mpart = base ? (float*)(base + o_bytes) : nullptr;
  p.Lpart = base ? (float*)(base + o_bytes + ml_bytes) : nullptr;
  p.lse = a.lse;
  char buf[320], part[64] = "";
  if (parts > 1) snprintf(part, sizeof part, ", each as %d ordered parts of %d", parts, p.kb_per * 64);
  snprintf(buf, sizeof buf, "attention: loop h [#tile<1>](%lld heads) x loop s [#sum softmax](%d key shards of %d%s) "
           "over %lld sequences, S=%lld, %s", (long long)a.H, a.Rkv, p.kb_per * 64 * parts, part, (long long)a.B,
           (long long)a.S, a.causal ? "causal" : "full");
  L.text = buf;
  plan.launches.push_back(L);
  if (a.Rkv > 1) {
    Launch C = L;
    C.kind = L_ATTN_COMBINE;
    C.name = "attn.combine";
    C.text = "attention_combine: O = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s, s ascending";
    plan.launches.push_back(C);
  }
}

// ---------------------------------------------------------------------------
// attention core backward
// ---------------------------------------------------------------------------
struct AttnBwdArgs {
  const void *Q = nullptr, *K = nullptr, *V = nullptr, *O = nullptr, *dO = nullptr;
  const float* lse = nullptr;
  void *dQ = nullptr, *dK = nullptr, *dV = nullptr;
  int64_t B = 0, S = 0, H = 0, dh = 0;
  int causal = 1;
  float scale = 0.f;
};

int validate_attn_bwd(const AttnBwdArgs& a, bool with_ptrs) {
  int st = validate_attn_shapes(a.B, a.S, a.H * a.dh, a.H, a.dh, 1, 1);
  if (st) return st;
  if (!with_ptrs || a.B * a.S == 0) return PARTIR_OK;
  if (!a.Q || !a.K || !a.V || !a.O || !a.dO || !a.lse || !a.dQ || !a.dK || !a.dV)
    return fail(PARTIR_E_NULL, "Q, K, V, O, dO, lse, dQ, dK and dV must be non-NULL");
  if (!aligned16(a.Q) || !aligned16(a.K) || !aligned16(a.V) || !aligned16(a.O) || !aligned16(a.dO) ||
      !aligned16(a.dQ) || !aligned16(a.dK) || !aligned16(a.dV) || ((uintptr_t)a.lse & 3))
    return fail(PARTIR_E_LAYOUT, "tensors must be 16-byte aligned (lse 4-byte)");
  return PARTIR_OK;
}

void plan_attn_bwd(const AttnBwdArgs& a, void* ws, Plan& plan) {
  const int64_t T = a.B * a.S, D = a.H * a.dh;
  plan.n_shards = 1;
  plan.n_tile_loops = 1;   // the heads loop
  const double pairs = a.causal ? (double)a.S * (a.S + 1) / 2 : (double)a.S * a.S;
  plan.flops = 2.5 * 4.0 * a.B * a.H * pairs * a.dh;   // dV, dP, dQ, dK and S: 5 products per pair
  if (T == 0) return;
  plan.ws_bytes = align_up((size_t)T * a.H * 4);
  Launch L;
  L.kind = L_ATTN_BWD;
  L.name = "attn.bwd";
  AttnBwdParams& p = L.attn_bwd;
  p.Q = (const uint16_t*)a.Q; p.K = (const uint16_t*)a.K; p.V = (const uint16_t*)a.V;
  p.O = (const uint16_t*)a.O; p.dO = (const uint16_t*)a.dO; p.lse = a.lse; p.Dstat = (float*)ws;
  p.dQ = (uint16_t*)a.dQ; p.dK = (uint16_t*)a.dK; p.dV = (uint16_t*)a.dV;
  p.ldq = p.ldk = p.ldv = p.ldo = p.ldg = p.lddq = p.lddk = p.lddv = D;
  p.B = (int)a.B; p.S = (int)a.S; p.H = (int)a.H; p.causal = a.causal;
  p.scale = a.scale > 0 ? a.scale : 1.0f / std::sqrt((float)a.dh);
  p.scale_log2 = p.scale * 1.4426950408889634f;
  char buf[256];
  snprintf(buf, sizeof buf, "attention_backward: loop h [#tile<1>](%lld heads) over %lld sequences, S=%lld, %s; "
           "dq pass (keys streamed) then dk/dv pass (queries streamed)", (long long)a.H, (long long)a.B,
           (long long)a.S, a.causal ? "causal" : "full");
  L.text = buf;
  plan.launches.push_back(L);
}

// ---------------------------------------------------------------------------
// attention block backward
// ---------------------------------------------------------------------------
struct AttnBlockBwdArgs {
  const void *X = nullptr, *Wq = nullptr, *Wk = nullptr, *Wv = nullptr, *Wo = nullptr;   // [fan_in, fan_out]
  const void* saved = nullptr;                                                         // from the training forward
  const void* dY = nullptr;
  void *dX = nullptr, *dWq = nullptr, *dWk = nullptr, *dWv = nullptr, *dWo = nullptr;
  int64_t B = 0, S = 0, D = 0, H = 0, dh = 0;
  int causal = 1;
  float scale = 0.f;
  int Rb = 1, Rm = 1;
};

int validate_attn_block_bwd(const AttnBlockBwdArgs& a, bool with_ptrs) {
  int st = validate_attn_shapes(a.B, a.S, a.D, a.H, a.dh, a.Rb, a.Rm);
  if (st) return st;
  if (!with_ptrs || a.B * a.S == 0) return PARTIR_OK;
  const void* ps[] = {a.X, a.Wq, a.Wk, a.Wv, a.Wo, a.saved, a.dY, a.dX, a.dWq, a.dWk, a.dWv, a.dWo};
  for (const void* q : ps) {
    if (!q) return fail(PARTIR_E_NULL, "every tensor must be non-NULL");
    if (!aligned16(q)) return fail(PARTIR_E_LAYOUT, "tensors must be 16-byte aligned");
  }
  return PARTIR_OK;
}

// Gradients of the attention block (same nest as partir_attn_block); every
// weight and its gradient is [fan_in, fan_out] = [D, D]:
//   dA = dY Wo^T                  loop b [#tile<0>] loop m [#tile<1>] (heads)
//   dQ|dK|dV = attention backward per head
//   dX = [dQ dK dV] [Wq Wk Wv]^T  loop b [#tile<0>] loop m [#sum], and the sum over q, k, v
//   dW{q,k,v} = X^T dQKV          loop m [#tile<1>] loop b [#sum]
//   dWo = A^T dY                  loop m [#tile<0>] loop b [#sum]
void plan_attn_block_bwd(const AttnBlockBwdArgs& a, void* ws, Plan& plan) {
  const int64_t T = a.B * a.S, D = a.D;
  plan.n_shards = a.Rb * a.Rm;
  plan.n_tile_loops = (a.Rb > 1) + 1;
  const double pairs = a.causal ? (double)a.S * (a.S + 1) / 2 : (double)a.S * a.S;
  plan.flops = 16.0 * T * D * D + 2.5 * 4.0 * a.B * a.H * pairs * a.dh;
  if (T == 0) return;
  const size_t dd = align_up((size_t)D * D * 2), td = align_up((size_t)T * D * 2);
  const size_t one = td;   // saved layout: Q | K | V | O | lse
  const char* sv = (const char*)a.saved;
  const void* Q = sv;
  const void* K = sv ? sv + one : nullptr;
  const void* V = sv ? sv + 2 * one : nullptr;
  const void* Ao = sv ? sv + 3 * one : nullptr;
  const float* lse = sv ? (const float*)(sv + 4 * one) : nullptr;
  char* base = (char*)ws;
  size_t off = 0;
  auto take = [&](size_t n) { char* p = base ? base + off : nullptr; off += n; return (void*)p; };
  void* dA = take(td);
  void* dQKV = take(3 * td);
  void* Dst = take(align_up((size_t)T * a.H * 4));
  void* part = base ? base + off : nullptr;
  // Every operand is read where it lies: the weights are the K-contiguous
  // transposed right operands of dA and dX, and the activations the [K, M] /
  // [K, N] operands of the weight gradients (no transposed copies).
  GemmSpec ga;
  ga.A = a.dY; ga.B[0] = a.Wo; ga.C[0] = dA;
  ga.lda = D; ga.ldb = D; ga.ldc = D; ga.M = T; ga.N = D; ga.K = D;
  ga.c_dtype = PARTIR_BF16; ga.rm = a.Rb; ga.rn = a.Rm;
  ga.name = "attn.bwd.da"; ga.label = "bwd.da dA = slice 0 dY[b] . (slice 0 Wo[m])^T";
  plan_gemm(ga, nullptr, plan);
  AttnBwdArgs c;
  c.Q = Q; c.K = K; c.V = V; c.O = Ao; c.dO = dA; c.lse = lse;
  c.dQ = dQKV; c.dK = dQKV ? (char*)dQKV + D * 2 : nullptr; c.dV = dQKV ? (char*)dQKV + 2 * D * 2 : nullptr;
  c.B = a.B; c.S = a.S; c.H = a.H; c.dh = a.dh; c.causal = a.causal; c.scale = a.scale;
  Plan core;
  plan_attn_bwd(c, Dst, core);
  Launch L = core.launches.back();
  L.attn_bwd.lddq = L.attn_bwd.lddk = L.attn_bwd.lddv = 3 * D;   // [dQ | dK | dV] side by side
  plan.launches.push_back(L);
  // dX: the right operand [Wq Wk Wv]^T is K-contiguous and split along K
  // over the three weights, read through a table of three K parts (whole-K
  // accumulation in q, k, v order)
  GemmSpec gx;
  gx.A = dQKV; gx.C[0] = a.dX;
  gx.lda = 3 * D; gx.ldb = D; gx.ldc = D; gx.M = T; gx.N = D; gx.K = 3 * D;
  gx.c_dtype = PARTIR_F32; gx.rm = a.Rb;
  gx.name = "attn.bwd.dx"; gx.label = "bwd.dx dX = sum over m and q|k|v of dQKV[b][:, m] . W{q,k,v}[:, m]^T";
  {
    const size_t first = plan.launches.size();
    plan_gemm(gx, part, plan);
    std::shared_ptr<GemmParts> t(new GemmParts{});
    t->b_nrows = (int)D; t->b_kcols = (int)D; t->b_nk = 3; t->b_gstride = 0;
    t->b[0] = (const uint16_t*)a.Wq; t->b[1] = (const uint16_t*)a.Wk; t->b[2] = (const uint16_t*)a.Wv;
    for (size_t i = first; i < plan.launches.size(); ++i) {
      Launch& L = plan.launches[i];
      L.kind = L.kind == L_GEMM_BF16_FIXUP ? L_GEMM_BF16_PARTS_FIXUP : L_GEMM_BF16_PARTS;
      L.parts = t;
      if (i == first) L.text += "; B^T read as K parts Wq | Wk | Wv";
    }
  }
  const char* wnames[3] = {"bwd.dwq dWq = sum_b (slice 0 X[b])^T . dQ[b][:, m]",
                           "bwd.dwk dWk = sum_b (slice 0 X[b])^T . dK[b][:, m]",
                           "bwd.dwv dWv = sum_b (slice 0 X[b])^T . dV[b][:, m]"};
  void* dW[3] = {a.dWq, a.dWk, a.dWv};
  for (int i = 0; i < 3; ++i) {
    GemmSpec gw;
    gw.A = a.X; gw.a_mn = true;
    gw.B[0] = dQKV ? (char*)dQKV + i * D * 2 : nullptr; gw.b_nk = 0; gw.C[0] = dW[i];
    gw.lda = D; gw.ldb = 3 * D; gw.ldc = D; gw.M = D; gw.N = D; gw.K = T;
    gw.c_dtype = PARTIR_F32; gw.rn = a.Rm; gw.rk = a.Rb; gw.sum_impl = PARTIR_SUM_FUSED;
    gw.name = "attn.bwd.dwqkv"; gw.label = wnames[i];
    plan_gemm(gw, nullptr, plan);
  }
  GemmSpec go;
  go.A = Ao; go.a_mn = true; go.B[0] = a.dY; go.b_nk = 0; go.C[0] = a.dWo;
  go.lda = D; go.ldb = D; go.ldc = D; go.M = D; go.N = D; go.K = T;
  go.c_dtype = PARTIR_F32; go.rm = a.Rm; go.rk = a.Rb;
  go.name = "attn.bwd.dwo"; go.label = "bwd.dwo dWo = sum_b A[b][:, m]^T . slice 0 dY[b]";
  plan_gemm(go, part, plan);
  plan.n_sum_loops = 4;
  plan.ws_bytes = off + std::max(gemm_ws_bytes(gx), gemm_ws_bytes(go));
}

// ---------------------------------------------------------------------------
// partir_mlp_block_backward
// ---------------------------------------------------------------------------
struct MlpBwdArgs {
  const void *X = nullptr, *W1 = nullptr, *b1 = nullptr, *W2 = nullptr, *dY = nullptr;
  const void* Z = nullptr;   // kept pre-activation; NULL: recomputed
  void *dX = nullptr, *dW1 = nullptr, *db1 = nullptr, *dW2 = nullptr, *db2 = nullptr;
  int64_t T, D, F;
  int act, Rb, Rm;
};

int validate_mlp_bwd(const MlpBwdArgs& a, bool with_ptrs) {
  if (a.T < 0 || a.D < 0 || a.F < 0) return fail(PARTIR_E_SHAPE, "T, D, F must be >= 0");
  if (a.T > (1 << 30) || a.D > (1 << 20) || a.F > (1 << 22) || a.T * std::max(a.D, a.F) > ((int64_t)1 << 37))
    return fail(PARTIR_E_SHAPE, "dims too large");
  if (a.Rb < 1 || a.Rm < 1) return fail(PARTIR_E_UNSUPPORTED, "R_batch and R_model must be >= 1");
  if (a.act != PARTIR_ACT_NONE && a.act != PARTIR_ACT_GELU_ERF) return fail(PARTIR_E_UNSUPPORTED, "act %d", a.act);
  if (a.T % a.Rb) return fail(PARTIR_E_DIVISIBILITY, "R_batch=%d does not divide T=%lld", a.Rb, (long long)a.T);
  if (a.F % a.Rm) return fail(PARTIR_E_DIVISIBILITY, "R_model=%d does not divide F=%lld", a.Rm, (long long)a.F);
  if (a.D % 8 || (a.F / a.Rm) % 8 || (a.T / a.Rb) % 8)
    return fail(PARTIR_E_LAYOUT, "D, F/R_model and T/R_batch must be multiples of 8 (16-byte runs; the weight "
                "gradients contract over tokens)");
  const bool live = a.T * a.D * a.F > 0;
  if (with_ptrs && live && (!a.X || !a.W1 || !a.W2 || !a.dY))
    return fail(PARTIR_E_NULL, "X, W1, W2 and dY must be non-NULL");
  if (with_ptrs && ((a.T * a.D > 0 && !a.dX) || (a.F * a.D > 0 && (!a.dW1 || !a.dW2))))
    return fail(PARTIR_E_NULL, "dX, dW1 and dW2 must be non-NULL when they hold elements");
  if (with_ptrs && a.db2 && a.T * a.D > 0 && !a.dY) return fail(PARTIR_E_NULL, "db2 needs dY");
  if (with_ptrs && (!aligned16(a.X) || !aligned16(a.W1) || !aligned16(a.W2) || !aligned16(a.dY) ||
                    !aligned16(a.dX) || !aligned16(a.dW1) || !aligned16(a.dW2) || !aligned16(a.b1) ||
                    !aligned16(a.db1) || !aligned16(a.db2) || !aligned16(a.Z)))
    return fail(PARTIR_E_LAYOUT, "tensors must be 16-byte aligned");
  return PARTIR_OK;
}

void plan_colsum(const void* in, void* partial, void* out, int64_t rows, int64_t cols, bool partial_ready,
                 const char* name, Plan& plan) {
  Launch L;
  L.kind = L_COLSUM;
  L.name = name;
  L.cs.in = (const uint16_t*)in; L.cs.partial = (float*)partial; L.cs.out = (float*)out;
  L.cs.ld = cols; L.cs.rows = (int)rows; L.cs.cols = (int)cols; L.cs.partial_ready = partial_ready;
  char buf[200];
  snprintf(buf, sizeof buf, "colsum: sum over %lld rows of [%lld,%lld], blocks of %d in order (the batch #sum of "
           "a bias gradient)%s", (long long)rows, (long long)rows, (long long)cols, kColSumChunk,
           partial_ready ? "; block sums from act_backward" : "");
  L.text = buf;
  plan.launches.push_back(L);
}

// Gradients of the Megatron MLP block (same nest as partir_mlp_block):
//   Z = X W1 + b1, H = act(Z), Y = H W2 + b2; given dY:
//   dH = dY W2^T     loop b [#tile<0>] loop m [#tile<1>]
//   dZ = dH * act'(Z)
//   dW2 = H^T dY     loop m [#tile<0>] loop b [#sum]   (the batch-parallel gradient reduction)
//   dW1 = X^T dZ     loop m [#tile<1>] loop b [#sum]
//   dX = dZ W1^T     loop b [#tile<0>] loop m [#sum]   (the model-parallel reduction)
//   db1 = sum_t dZ, db2 = sum_t dY
// Weights and their gradients are [fan_in, fan_out]: W1, dW1 [D, F]; W2, dW2 [F, D].
void plan_mlp_bwd(const MlpBwdArgs& a, void* ws, Plan& plan) {
  const int64_t T = a.T, D = a.D, F = a.F;
  plan.n_shards = a.Rb * a.Rm;
  plan.n_tile_loops = 2;
  plan.flops = 10.0 * T * D * F;          // Z recomputed (2TDF) + dH, dW2, dW1, dX (8TDF)
  if (T == 0 && D == 0 && F == 0) return;
  const bool live = T * D * F > 0;
  // without a contraction only the bias-gradient column sums use the workspace
  const size_t tf = live ? align_up((size_t)T * F * 2) : 0, td = live ? align_up((size_t)T * D * 2) : 0,
               df = live ? align_up((size_t)D * F * 2) : 0;
  const size_t cs_bytes =
      (a.db1 || a.db2) ? align_up((size_t)((T + kColSumChunk - 1) / kColSumChunk) * std::max(D, F) * 4) : 0;
  char* base = (char*)ws;
  size_t off = 0;
  auto take = [&](size_t n) { char* p = base ? base + off : nullptr; off += n; return (void*)p; };
  void* Z = a.Z ? (void*)a.Z : take(tf);
  void* dH = take(tf);
  void* dZ = take(tf);
  void* H = take(tf);
  void* csp = take(cs_bytes);
  void* part = base ? base + off : nullptr;
  // Every operand is read where it lies: W1 is the [K, N] right operand of
  // Z and, K-contiguous, the transposed right operand of dX (W2 likewise of
  // dH); the activations are the [K, M] / [K, N] operands of the weight
  // gradients (no transposed copies).
  GemmSpec gz, gh, g2, g1, gx;
  if (live) {
    if (!a.Z) {
      gz.A = a.X; gz.B[0] = a.W1; gz.b_nk = 0; gz.C[0] = Z; gz.bias[0] = (const float*)a.b1;
      gz.lda = D; gz.ldb = F; gz.ldc = F; gz.M = T; gz.N = F; gz.K = D;
      gz.c_dtype = PARTIR_BF16; gz.rm = a.Rb; gz.rn = a.Rm;
      gz.name = "mlp.bwd.z"; gz.label = "bwd.z  Z = slice 0 X[b] . slice 1 W1[m] (recomputed)";
      plan_gemm(gz, nullptr, plan);
    }
    gh.A = a.dY; gh.B[0] = a.W2; gh.C[0] = dH;
    gh.lda = D; gh.ldb = D; gh.ldc = F; gh.M = T; gh.N = F; gh.K = D;
    gh.c_dtype = PARTIR_BF16; gh.rm = a.Rb; gh.rn = a.Rm;
    gh.name = "mlp.bwd.dh"; gh.label = "bwd.dh dH = slice 0 dY[b] . (slice 0 W2[m])^T";
    plan_gemm(gh, nullptr, plan);
    Launch E;
    E.kind = L_ACT_BWD;
    E.name = "mlp.bwd.act";
    E.act.Z = (const uint16_t*)Z; E.act.dH = (const uint16_t*)dH; E.act.dZ = (uint16_t*)dZ;
    E.act.H = (uint16_t*)H; E.act.ld = F;
    E.act.colpart = a.db1 ? (float*)csp : nullptr;   // db1's block sums, fused
    E.act.rows = (int)T; E.act.cols = (int)F; E.act.act = a.act;
    E.text = a.act ? "act_backward: dZ = dH * gelu'(Z); H = gelu(Z)" : "act_backward: dZ = dH; H = Z";
    plan.launches.push_back(E);
    g2.A = H; g2.a_mn = true; g2.B[0] = a.dY; g2.b_nk = 0; g2.C[0] = a.dW2;
    g2.lda = F; g2.ldb = D; g2.ldc = D; g2.M = F; g2.N = D; g2.K = T;
    g2.ab_dtype = PARTIR_BF16; g2.c_dtype = PARTIR_F32; g2.rm = a.Rm; g2.rk = a.Rb;
    g2.name = "mlp.bwd.dw2"; g2.label = "bwd.dw2 dW2 = sum_b H[b][:, m]^T . slice 0 dY[b]";
    plan_gemm(g2, part, plan);
    g1.A = a.X; g1.a_mn = true; g1.B[0] = dZ; g1.b_nk = 0; g1.C[0] = a.dW1;
    g1.lda = D; g1.ldb = F; g1.ldc = F; g1.M = D; g1.N = F; g1.K = T;
    g1.c_dtype = PARTIR_F32; g1.rn = a.Rm; g1.rk = a.Rb;
    g1.name = "mlp.bwd.dw1"; g1.label = "bwd.dw1 dW1 = sum_b (slice 0 X[b])^T . dZ[b][:, m]";
    plan_gemm(g1, part, plan);
    gx.A = dZ; gx.B[0] = a.W1; gx.C[0] = a.dX;
    gx.lda = F; gx.ldb = F; gx.ldc = D; gx.M = T; gx.N = D; gx.K = F;
    gx.c_dtype = PARTIR_F32; gx.rm = a.Rb; gx.rk = a.Rm;
    gx.name = "mlp.bwd.dx"; gx.label = "bwd.dx dX = sum_m dZ[b][:, m] . (slice 1 W1[m])^T";
    plan_gemm(gx, part, plan);
    plan.n_sum_loops = 3;
    // db1 from act_backward's block sums (before anything reuses csp), then db2
    if (a.db1) plan_colsum(dZ, csp, a.db1, T, F, true, "mlp.bwd.db", plan);
    if (a.db2) plan_colsum(a.dY, csp, a.db2, T, D, false, "mlp.bwd.db", plan);
  } else {
    // an empty dim: every gradient that still has elements is an empty sum
    // (zeros), except db2 = sum_t dY when only F is 0
    if (T * D > 0) plan_empty_sum(a.dX, T, D, D, false, nullptr, nullptr, 0, false, "mlp.bwd.dx", plan);
    if (F * D > 0) {
      plan_empty_sum(a.dW1, D, F, F, false, nullptr, nullptr, 0, false, "mlp.bwd.dw1", plan);
      plan_empty_sum(a.dW2, F, D, D, false, nullptr, nullptr, 0, false, "mlp.bwd.dw2", plan);
    }
    if (a.db1 && F > 0) plan_empty_sum(a.db1, 1, F, F, false, nullptr, nullptr, 0, false, "mlp.bwd.db", plan);
    if (a.db2 && D > 0) plan_colsum(a.dY, csp, a.db2, T, D, false, "mlp.bwd.db", plan);
  }
  size_t gws = 0;
  if (live) gws = std::max({gemm_ws_bytes(g2), gemm_ws_bytes(g1), gemm_ws_bytes(gx)});
  plan.ws_bytes = off + gws;
}

void fill_info(const Plan& plan, partir_plan_info* info) {
  if (!info) return;
  info->n_virtual_shards = plan.n_shards;
  info->n_tile_loops = plan.n_tile_loops;
  info->n_sum_loops = plan.n_sum_loops;
  info->n_sum_splitk = plan.n_sum_splitk;
  info->n_launches = (int)plan.launches.size();
  info->reserved = 0;
  info->workspace_bytes = plan.ws_bytes;
  info->flops = plan.flops;
}

}  // namespace

void set_last_error(const std::string& msg) { g_error = msg; }

// partir_loop_matmul's argument checks alone (pointers included), for the
// no-allocation variant, which must report them before it touches a device.
int validate_loop_matmul_call(const void* A, const void* B, void* C, int64_t M, int64_t N, int64_t K,
                              int64_t lda, int64_t ldb, int64_t ldc, int ab_dtype, int c_dtype, int b_layout,
                              int tile_axis, int sum_axis, int R, int sum_impl) {
  MatmulArgs a{A, B, C, M, N, K, lda, ldb, ldc, ab_dtype, c_dtype, b_layout, tile_axis, sum_axis, R, sum_impl};
  return validate_matmul(a, true);
}

}  // namespace partir

using namespace partir;

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* partir_status_string(int status) {
  switch (status) {
    case PARTIR_OK: return "PARTIR_OK";
    case PARTIR_E_NULL: return "PARTIR_E_NULL";
    case PARTIR_E_SHAPE: return "PARTIR_E_SHAPE";
    case PARTIR_E_DIVISIBILITY: return "PARTIR_E_DIVISIBILITY";
    case PARTIR_E_AXIS: return "PARTIR_E_AXIS";
    case PARTIR_E_DTYPE: return "PARTIR_E_DTYPE";
    case PARTIR_E_LAYOUT: return "PARTIR_E_LAYOUT";
    case PARTIR_E_WORKSPACE: return "PARTIR_E_WORKSPACE";
    case PARTIR_E_HIP: return "PARTIR_E_HIP";
    case PARTIR_E_UNSUPPORTED: return "PARTIR_E_UNSUPPORTED";
    default: return "PARTIR_E_UNKNOWN";
  }
}

const char* partir_last_error(void) { return g_error.c_str(); }
const char* partir_version(void) { return "libpartir 0.1 (gfx950)"; }
const char* partir_last_plan_text(void) { return g_plan_text.c_str(); }

// ---- loop_matmul ----------------------------------------------------------------
size_t partir_loop_matmul_workspace(int64_t M, int64_t N, int64_t K, int ab_dtype, int c_dtype,
                                    int b_layout, int tile_axis, int sum_axis, int R, int sum_impl) {
  MatmulArgs a{nullptr, nullptr, nullptr, M, N, K,
               K, b_layout == PARTIR_B_KN ? N : K, N, ab_dtype, c_dtype, b_layout, tile_axis, sum_axis, R, sum_impl};
  a.lda = ((K + 7) / 8) * 8;
  a.ldb = b_layout == PARTIR_B_KN ? ((N + 7) / 8) * 8 : a.lda;
  a.ldc = ((N + 7) / 8) * 8;
  if (validate_matmul(a, false) != PARTIR_OK) return (size_t)-1;
  return gemm_ws_bytes(matmul_spec(a));
}

int partir_plan_loop_matmul(int64_t M, int64_t N, int64_t K, int ab_dtype, int c_dtype, int b_layout,
                            int tile_axis, int sum_axis, int R, int sum_impl, partir_plan_info* info) {
  MatmulArgs a{nullptr, nullptr, nullptr, M, N, K, 0, 0, 0, ab_dtype, c_dtype, b_layout, tile_axis, sum_axis, R, sum_impl};
  a.lda = ((K + 7) / 8) * 8;
  a.ldb = b_layout == PARTIR_B_KN ? ((N + 7) / 8) * 8 : a.lda;
  a.ldc = ((N + 7) / 8) * 8;
  int st = validate_matmul(a, false);
  if (st) return st;
  Plan plan;
  plan_matmul(a, nullptr, plan);
  keep_plan_text(plan, "loop_matmul");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_loop_matmul(const void* A, const void* B, void* C, int64_t M, int64_t N, int64_t K,
                       int64_t lda, int64_t ldb, int64_t ldc, int ab_dtype, int c_dtype, int b_layout,
                       int tile_axis, int sum_axis, int R, int sum_impl, void* ws, size_t ws_bytes, void* stream) {
  MatmulArgs a{A, B, C, M, N, K, lda, ldb, ldc, ab_dtype, c_dtype, b_layout, tile_axis, sum_axis, R, sum_impl};
  int st = validate_matmul(a, true);
  if (st) return st;
  Plan plan;
  plan_matmul(a, ws, plan);
  if ((st = check_ws(plan, ws, ws_bytes))) return st;
  keep_plan_text(plan, "loop_matmul");
  return execute(plan, stream);
}

// ---- mlp_block -------------------------------------------------------------------
size_t partir_mlp_block_workspace(int64_t T, int64_t D, int64_t F, int out_dtype, int R_batch, int R_model) {
  MlpArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, T, D, F, PARTIR_BF16, out_dtype, PARTIR_ACT_GELU_ERF, R_batch, R_model};
  if (validate_mlp(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_mlp(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_mlp_block(int64_t T, int64_t D, int64_t F, int out_dtype, int R_batch, int R_model,
                          partir_plan_info* info) {
  MlpArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, T, D, F, PARTIR_BF16, out_dtype, PARTIR_ACT_GELU_ERF, R_batch, R_model};
  int st = validate_mlp(a, false);
  if (st) return st;
  Plan plan;
  plan_mlp(a, nullptr, plan);
  keep_plan_text(plan, "mlp_block");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_mlp_block(const void* X, const void* W1, const void* b1, const void* W2, const void* b2, void* Y,
                     int64_t T, int64_t D, int64_t F, int in_dtype, int out_dtype, int act,
                     int R_batch, int R_model, void* ws, size_t ws_bytes, void* stream) {
  MlpArgs a{X, W1, b1, W2, b2, Y, T, D, F, in_dtype, out_dtype, act, R_batch, R_model};
  int st = validate_mlp(a, true);
  if (st) return st;
  Plan probe;
  plan_mlp(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_mlp(a, ws, plan);
  keep_plan_text(plan, "mlp_block");
  return execute(plan, stream);
}

int partir_mlp_block_train(const void* X, const void* W1, const void* b1, const void* W2, const void* b2,
                           void* Y, void* Z, int64_t T, int64_t D, int64_t F, int in_dtype, int out_dtype,
                           int act, int R_batch, int R_model, void* ws, size_t ws_bytes, void* stream) {
  MlpArgs a{X, W1, b1, W2, b2, Y, T, D, F, in_dtype, out_dtype, act, R_batch, R_model, Z};
  if (T * D * F > 0 && !Z) return fail(PARTIR_E_NULL, "Z must be non-NULL (unless empty)");
  int st = validate_mlp(a, true);
  if (st) return st;
  Plan probe;
  plan_mlp(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_mlp(a, ws, plan);
  keep_plan_text(plan, "mlp_block_train");
  return execute(plan, stream);
}

// ---- MLP block on device-local arrays (BP + MP + Z3, activations sharded on M) ------
// Device (b, m) of the mesh {B: R_batch, M: R_model} is part index b * R_model + m.
namespace {
struct MlpShardedArgs {
  const void* const* X = nullptr;     // [T/(RB RM), D] per device
  const void* const* W1t = nullptr;   // W1t[F/RM rows m, D/RB cols b] per device
  const void* b1 = nullptr;
  const void* const* W2t = nullptr;   // W2t[D/RB rows b, F/RM cols m] per device
  const void* b2 = nullptr;
  void* const* Y = nullptr;           // [T/(RB RM), D] per device
  int64_t T = 0, D = 0, F = 0;
  int out = PARTIR_F32, act = PARTIR_ACT_GELU_ERF, Rb = 1, Rm = 1;
};

int validate_mlp_sharded(const MlpShardedArgs& a, bool with_ptrs) {
  if (a.T < 0 || a.D < 0 || a.F < 0) return fail(PARTIR_E_SHAPE, "T, D, F must be >= 0");
  if (a.T > (1 << 30) || a.D > (1 << 20) || a.F > (1 << 22)) return fail(PARTIR_E_SHAPE, "dims too large");
  if (a.Rb < 1 || a.Rm < 1) return fail(PARTIR_E_UNSUPPORTED, "R_batch and R_model must be >= 1");
  const int nd = a.Rb * a.Rm;
  if (nd > kMaxParts) return fail(PARTIR_E_UNSUPPORTED, "at most %d devices (R_batch * R_model)", kMaxParts);
  if (!valid_dtype(a.out)) return fail(PARTIR_E_DTYPE, "out_dtype must be F32 or BF16");
  if (a.act != PARTIR_ACT_NONE && a.act != PARTIR_ACT_GELU_ERF) return fail(PARTIR_E_UNSUPPORTED, "act %d", a.act);
  if (a.T % nd) return fail(PARTIR_E_DIVISIBILITY, "R_batch*R_model=%d does not divide T=%lld", nd, (long long)a.T);
  if (a.D % a.Rb) return fail(PARTIR_E_DIVISIBILITY, "R_batch=%d does not divide D=%lld", a.Rb, (long long)a.D);
  if (a.F % a.Rm) return fail(PARTIR_E_DIVISIBILITY, "R_model=%d does not divide F=%lld", a.Rm, (long long)a.F);
  if ((a.T / nd) % 64 || (a.D / a.Rb) % 64 || (a.F / a.Rm) % 64)
    return fail(PARTIR_E_LAYOUT, "T/(R_batch R_model), D/R_batch and F/R_model must be multiples of 64 (the "
                "GEMM's 64-row load blocks and 64-wide K tiles never straddle two arrays)");
  if (!with_ptrs) return PARTIR_OK;
  const bool live = a.T * a.D * a.F > 0, out_live = a.T * a.D > 0;
  if ((live && (!a.X || !a.W1t || !a.W2t)) || (out_live && !a.Y))
    return fail(PARTIR_E_NULL, "the part arrays must be non-NULL");
  if (!aligned16(a.b1) || !aligned16(a.b2)) return fail(PARTIR_E_LAYOUT, "b1, b2 must be 16-byte aligned");
  for (int i = 0; i < nd; ++i) {
    if (live && (!a.X[i] || !a.W1t[i] || !a.W2t[i])) return fail(PARTIR_E_NULL, "part %d is NULL", i);
    if (out_live && !a.Y[i]) return fail(PARTIR_E_NULL, "output part %d is NULL", i);
    if ((live && (!aligned16(a.X[i]) || !aligned16(a.W1t[i]) || !aligned16(a.W2t[i]))) ||
        (out_live && !aligned16(a.Y[i])))
      return fail(PARTIR_E_LAYOUT, "part %d is not 16-byte aligned", i);
  }
  return PARTIR_OK;
}

// The lowered program of the MLP under BP + MP + Z3 with its activations
// sharded on M (Sec. 3's FSDP chain and the remark after it; Sec. 6's
// collectives): per device (b, m)
//   x  = all_gather<M, dim 0>(X_bm)               -> up GEMM's A rows, read in place
//   w1 = all_gather<B, dim 0 of W1>(W1_bm)        -> up GEMM's B K-blocks, read in place
//   h  = act(x w1 + b1_m)                         -> H[b rows, m cols] (workspace)
//   w2 = all_gather<B, dim 1 of W2>(W2_bm)        -> down GEMM's B row blocks, read in place
//   y  = reduce_scatter<M, dim 0>(h w2) + b2      -> the down GEMM's fused #sum over m, each
//                                                    row block stored by its owner into Y_bm
void plan_mlp_sharded(const MlpShardedArgs& a, void* ws, Plan& plan) {
  const int nd = a.Rb * a.Rm;
  const int64_t T = a.T, D = a.D, F = a.F, rows_dev = T / nd;
  plan.n_shards = nd;
  plan.n_tile_loops = (a.Rb > 1) + 1;
  plan.flops = 4.0 * T * D * F;
  if (T * D == 0) return;
  if (F == 0) {   // every model shard is empty: each device's slice is b2
    plan.n_sum_loops = 1;
    for (int i = 0; i < nd; ++i)
      plan_empty_sum(a.Y ? a.Y[i] : nullptr, rows_dev, D, D, a.out == PARTIR_BF16, (const float*)a.b2, nullptr,
                     0, false, "mlp.down", plan);
    return;
  }
  void* H = ws;
  plan.ws_bytes = align_up((size_t)T * F * 2);
  auto parted = [&](const GemmSpec& g, GemmParts* t, const char* how) {
    plan_gemm(g, nullptr, plan);
    Launch& L = plan.launches.back();
    L.kind = L_GEMM_BF16_PARTS;
    L.parts.reset(t);
    L.text += how;
  };
  GemmSpec g1;
  g1.A = nullptr; g1.B[0] = nullptr; g1.C[0] = H; g1.bias[0] = (const float*)a.b1;
  g1.lda = D; g1.ldb = D / a.Rb; g1.ldc = F;
  g1.M = T; g1.N = F; g1.K = D;
  g1.c_dtype = PARTIR_BF16; g1.rm = a.Rb; g1.rn = a.Rm; g1.act = a.act;
  g1.name = "mlp.up";
  g1.label = "mlp.up   H = act(all_gather<M>(X)[b] . all_gather<B>(W1)[:, m])";
  GemmParts* t1 = new GemmParts{};
  t1->a_rows = (int)rows_dev;
  t1->b_nrows = (int)(F / a.Rm); t1->b_kcols = (int)(D / a.Rb); t1->b_nk = a.Rb;
  for (int b = 0; b < a.Rb; ++b)
    for (int m = 0; m < a.Rm; ++m) {
      const int dev = b * a.Rm + m;
      if (a.X) t1->a[dev] = (const uint16_t*)a.X[dev];
      if (a.W1t) t1->b[m * a.Rb + b] = (const uint16_t*)a.W1t[dev];   // N block m, K block b
    }
  parted(g1, t1, "; X rows and W1 blocks read from each device's array (fused all_gathers)");
  GemmSpec g2;
  g2.A = H; g2.B[0] = nullptr; g2.C[0] = nullptr; g2.bias[0] = (const float*)a.b2;
  g2.lda = F; g2.ldb = F / a.Rm; g2.ldc = D;
  g2.M = T; g2.N = D; g2.K = F;
  g2.c_dtype = a.out; g2.rm = a.Rb; g2.rk = a.Rm; g2.sum_impl = PARTIR_SUM_FUSED;
  g2.name = "mlp.down";
  g2.label = "mlp.down Y = reduce_scatter<M>(sum_m H[:, m] . all_gather<B>(W2)[m, :])";
  GemmParts* t2 = new GemmParts{};
  t2->b_nrows = (int)(D / a.Rb); t2->b_kcols = (int)(F / a.Rm); t2->b_nk = a.Rm;
  t2->c_rows = (int)rows_dev;
  for (int i = 0; i < nd; ++i) {
    if (a.W2t) t2->b[i] = (const uint16_t*)a.W2t[i];   // device (b, m): N block b, K block m
    if (a.Y) t2->c[i] = a.Y[i];
  }
  parted(g2, t2, "; W2 blocks read in place; each row block stored by its owner (fused reduce_scatter)");
}
}  // namespace

// ---- decoder layer on device-local arrays (BP + MP + Z3, sequence-parallel norms) --
namespace {
struct DecShardedArgs {
  void* const* x = nullptr;                 // [T/(RB RM), D] fp32 per device, updated in place
  const void *g1 = nullptr, *g2 = nullptr;
  float eps = 1e-6f;
  const void* const* W[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};   // q, k, v, o, 1, 2
  int64_t B = 0, S = 0, D = 0, H = 0, dh = 0, F = 0;
  int Rb = 1, Rm = 1;
};

int validate_dec_sharded(const DecShardedArgs& a, bool with_ptrs) {
  int st = validate_attn_shapes(a.B, a.S, a.D, a.H, a.dh, a.Rb, a.Rm);
  if (st) return st;
  const int nd = a.Rb * a.Rm;
  const int64_t T = a.B * a.S;
  // the Q|K|V projection reads three weights' blocks through one part table
  if (3 * nd > kMaxParts)
    return fail(PARTIR_E_UNSUPPORTED, "at most %d devices (R_batch * R_model) for the decoder layer", kMaxParts / 3);
  if (a.F < 0 || a.F > (1 << 22)) return fail(PARTIR_E_SHAPE, "F out of range");
  if (!(a.eps >= 0.0f)) return fail(PARTIR_E_SHAPE, "eps must be >= 0");
  if (a.F % a.Rm) return fail(PARTIR_E_DIVISIBILITY, "R_model=%d does not divide F=%lld", a.Rm, (long long)a.F);
  if (a.D % a.Rb) return fail(PARTIR_E_DIVISIBILITY, "R_batch=%d does not divide D=%lld", a.Rb, (long long)a.D);
  if (T % nd) return fail(PARTIR_E_DIVISIBILITY, "R_batch*R_model=%d does not divide T=%lld", nd, (long long)T);
  if ((T / nd) % 16 || (a.D / a.Rb) % 64 || (a.F / a.Rm) % 64)
    return fail(PARTIR_E_LAYOUT, "T/(R_batch R_model) must be a multiple of 16 and D/R_batch, F/R_model of 64");
  if (!with_ptrs || T == 0) return PARTIR_OK;
  if (!a.x || !a.g1 || (a.F > 0 && !a.g2)) return fail(PARTIR_E_NULL, "x parts, g1 and g2 must be non-NULL");
  if (!aligned16(a.g1) || !aligned16(a.g2)) return fail(PARTIR_E_LAYOUT, "g1, g2 must be 16-byte aligned");
  for (int w = 0; w < 6; ++w) {
    if (w >= 4 && a.F == 0) continue;
    if (!a.W[w]) return fail(PARTIR_E_NULL, "weight part arrays must be non-NULL");
  }
  for (int i = 0; i < nd; ++i) {
    if (!a.x[i]) return fail(PARTIR_E_NULL, "x part %d is NULL", i);
    if (!aligned16(a.x[i])) return fail(PARTIR_E_LAYOUT, "x part %d is not 16-byte aligned", i);
    for (int w = 0; w < 6; ++w) {
      if (w >= 4 && a.F == 0) continue;
      if (!a.W[w][i]) return fail(PARTIR_E_NULL, "weight part %d is NULL", i);
      if (!aligned16(a.W[w][i])) return fail(PARTIR_E_LAYOUT, "weight part %d is not 16-byte aligned", i);
    }
  }
  return PARTIR_OK;
}

// The decoder layer's lowered program on device-local arrays, per device
// (b, m): the RMSNorms on the device's own tokens write into the gathered
// activation buffer (the all_gather over M fused into the norm's store); the
// projections read the Z3 weight parts in place (all_gathers over B); the
// out-projection and FFN-down #sums over m are accumulated in the tile and
// each row block is added into its owner's residual part (reduce_scatter
// fused with the residual add).
void plan_dec_sharded(const DecShardedArgs& a, void* ws, Plan& plan) {
  const int nd = a.Rb * a.Rm;
  const int64_t T = a.B * a.S, D = a.D, F = a.F, rows_dev = T / nd;
  plan.n_shards = nd;
  plan.n_tile_loops = (a.Rb > 1) + 2;
  plan.flops = 8.0 * T * D * D + 4.0 * a.B * a.H * ((double)a.S * (a.S + 1) / 2) * a.dh + 4.0 * T * D * F;
  if (T == 0) return;
  char* base = (char*)ws;
  const size_t xn_bytes = align_up((size_t)T * D * 2);
  const size_t core = attn_core_bytes(T, D);
  const size_t h_bytes = align_up((size_t)T * F * 2);
  char* xn = base;
  char* qkvo = base ? base + xn_bytes : nullptr;
  char* Hf = base ? base + xn_bytes + core : nullptr;
  char* gws = base ? base + xn_bytes + core + (F > 0 ? h_bytes : 0) : nullptr;   // tail parts, one GEMM at a time
  const size_t one = align_up((size_t)T * D * 2);
  // the four GEMMs: Q|K|V (three groups), attention out, FFN up, FFN down
  GemmSpec gq;
  gq.A = xn;
  for (int i = 0; i < 3; ++i) gq.C[i] = qkvo ? qkvo + i * one : nullptr;
  gq.ngroups = 3;
  gq.lda = D; gq.ldb = D / a.Rb; gq.ldc = D; gq.M = T; gq.N = D; gq.K = D;
  gq.c_dtype = PARTIR_BF16; gq.rm = a.Rb; gq.rn = a.Rm; gq.tail_ok = true;
  gq.name = "attn.qkv"; gq.label = "attn.qkv Q|K|V = xn[b] . all_gather<B>(W{q,k,v})[:, m]";
  GemmSpec go;
  go.A = qkvo ? qkvo + 3 * one : nullptr; go.resid_add = true;
  go.lda = D; go.ldb = D / a.Rm; go.ldc = D; go.M = T; go.N = D; go.K = D;
  go.c_dtype = PARTIR_F32; go.rm = a.Rb; go.rk = a.Rm; go.sum_impl = PARTIR_SUM_FUSED; go.tail_ok = true;
  go.name = "attn.out"; go.label = "dec.attn_out x_bm += reduce_scatter<M>(sum_m O[:, m] . all_gather<B>(Wo)[m])";
  GemmSpec g1;
  g1.A = xn; g1.C[0] = Hf;
  g1.lda = D; g1.ldb = D / a.Rb; g1.ldc = F; g1.M = T; g1.N = F; g1.K = D;
  g1.c_dtype = PARTIR_BF16; g1.rm = a.Rb; g1.rn = a.Rm; g1.act = 1;
  g1.name = "mlp.up"; g1.label = "dec.ffn_up H = gelu(hn[b] . all_gather<B>(W1)[:, m])";
  GemmSpec g2;
  g2.A = Hf; g2.resid_add = true;
  g2.lda = F; g2.ldb = F / a.Rm; g2.ldc = D; g2.M = T; g2.N = D; g2.K = F;
  g2.c_dtype = PARTIR_F32; g2.rm = a.Rb; g2.rk = a.Rm; g2.sum_impl = PARTIR_SUM_FUSED; g2.tail_ok = true;
  g2.name = "mlp.down"; g2.label = "dec.ffn_down x_bm += reduce_scatter<M>(sum_m H[:, m] . all_gather<B>(W2)[m])";
  plan.ws_bytes = xn_bytes + core + std::max(gemm_ws_bytes(gq), gemm_ws_bytes(go));
  if (F > 0) plan.ws_bytes = xn_bytes + core + h_bytes +
                             std::max({gemm_ws_bytes(gq), gemm_ws_bytes(go), gemm_ws_bytes(g1), gemm_ws_bytes(g2)});
  auto norms = [&](const void* g) {
    // one launch over every device's tokens: each row is normalised where it
    // lives and stored into the gathered buffer
    plan_rmsnorm(nullptr, (const float*)g, xn, T, D, a.eps, a.Rb, plan);
    Launch& L = plan.launches.back();
    L.kind = L_RMS_PARTS;
    RmsParts* t = new RmsParts{};
    t->rows_part = (int)rows_dev;
    for (int i = 0; i < nd; ++i) t->x[i] = a.x ? (const float*)a.x[i] : nullptr;
    L.rms_parts.reset(t);
    char buf[200];
    snprintf(buf, sizeof buf, "rmsnorm: %d devices x %lld tokens x %lld, each device's own tokens (sequence-parallel), "
             "stored into the gathered buffer (all_gather<M>)", nd, (long long)rows_dev, (long long)D);
    L.text = buf;
  };
  // B part table of column-parallel weights W^T [out, in] (one group per
  // weight): part (b, m) holds rows block m, cols block b -> N block m, K block b
  auto col_parts = [&](const void* const* const* W, int ng, int64_t n_out) {
    GemmParts* t = new GemmParts{};
    t->b_nrows = (int)(n_out / a.Rm); t->b_kcols = (int)(D / a.Rb); t->b_nk = a.Rb; t->b_gstride = nd;
    for (int g = 0; g < ng; ++g)
      for (int b = 0; b < a.Rb; ++b)
        for (int m = 0; m < a.Rm; ++m)
          t->b[g * nd + m * a.Rb + b] = W[g] ? (const uint16_t*)W[g][b * a.Rm + m] : nullptr;
    return t;
  };
  // row-parallel weight W^T [D, in]: part (b, m) = rows block b, cols block m;
  // the output rows go into the residual parts
  auto row_parts = [&](const void* const* W, int64_t k_in) {
    GemmParts* t = new GemmParts{};
    t->b_nrows = (int)(D / a.Rb); t->b_kcols = (int)(k_in / a.Rm); t->b_nk = a.Rm;
    t->c_rows = (int)rows_dev;
    for (int i = 0; i < nd; ++i) {
      t->b[i] = W ? (const uint16_t*)W[i] : nullptr;
      t->c[i] = a.x ? a.x[i] : nullptr;
    }
    return t;
  };
  // one GEMM's launches (main and, with a split last wave, its fixup) on the
  // device-local arrays of `t`
  auto parted = [&](const GemmSpec& g, GemmParts* t, const char* how) {
    const size_t first = plan.launches.size();
    plan_gemm(g, gws, plan);
    std::shared_ptr<GemmParts> sp(t);
    for (size_t i = first; i < plan.launches.size(); ++i) {
      Launch& L = plan.launches[i];
      L.kind = L.kind == L_GEMM_BF16_FIXUP ? L_GEMM_BF16_PARTS_FIXUP : L_GEMM_BF16_PARTS;
      L.parts = sp;
      if (i == first) L.text += how;
    }
  };
  norms(a.g1);
  const void* const* wqkv[3] = {a.W[0], a.W[1], a.W[2]};
  parted(gq, col_parts(wqkv, 3, D), "; weight blocks read in place (fused all_gather)");
  plan_attention_launch(qkvo, a.B, a.S, D, a.H, a.dh, 1, 0.0f, a.Rm, plan, nullptr);
  parted(go, row_parts(a.W[3], D), "; each row block added into its owner's residual part (fused reduce_scatter)");
  plan.n_sum_loops = 1;
  if (F == 0) return;   // an FFN of width 0 adds the empty sum: x is unchanged
  norms(a.g2);
  const void* const* w1[1] = {a.W[4]};
  parted(g1, col_parts(w1, 1, F), "; weight blocks read in place (fused all_gather)");
  parted(g2, row_parts(a.W[5], F), "; each row block added into its owner's residual part (fused reduce_scatter)");
  plan.n_sum_loops = 2;
}
}  // namespace

size_t partir_decoder_layer_sharded_workspace(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                                              int64_t F, int R_batch, int R_model) {
  DecShardedArgs a;
  a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.F = F; a.Rb = R_batch; a.Rm = R_model;
  if (validate_dec_sharded(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_dec_sharded(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_decoder_layer_sharded(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head, int64_t F,
                                      int R_batch, int R_model, partir_plan_info* info) {
  DecShardedArgs a;
  a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.F = F; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_dec_sharded(a, false);
  if (st) return st;
  Plan plan;
  plan_dec_sharded(a, nullptr, plan);
  keep_plan_text(plan, "decoder_layer_sharded");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_decoder_layer_sharded(void* const* x_parts, const void* g1, const void* g2, float eps,
                                 const void* const* Wq_parts, const void* const* Wk_parts,
                                 const void* const* Wv_parts, const void* const* Wo_parts,
                                 const void* const* W1_parts, const void* const* W2_parts, int64_t B, int64_t S,
                                 int64_t D, int64_t n_heads, int64_t d_head, int64_t F, int R_batch, int R_model,
                                 void* ws, size_t ws_bytes, void* stream) {
  DecShardedArgs a;
  a.x = x_parts; a.g1 = g1; a.g2 = g2; a.eps = eps;
  a.W[0] = Wq_parts; a.W[1] = Wk_parts; a.W[2] = Wv_parts; a.W[3] = Wo_parts; a.W[4] = W1_parts; a.W[5] = W2_parts;
  a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.F = F; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_dec_sharded(a, true);
  if (st) return st;
  Plan probe;
  plan_dec_sharded(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_dec_sharded(a, ws, plan);
  keep_plan_text(plan, "decoder_layer_sharded");
  return execute(plan, stream);
}

size_t partir_mlp_block_sharded_workspace(int64_t T, int64_t D, int64_t F, int R_batch, int R_model) {
  MlpShardedArgs a;
  a.T = T; a.D = D; a.F = F; a.Rb = R_batch; a.Rm = R_model;
  if (validate_mlp_sharded(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_mlp_sharded(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_mlp_block_sharded(int64_t T, int64_t D, int64_t F, int act, int R_batch, int R_model,
                                  partir_plan_info* info) {
  MlpShardedArgs a;
  a.T = T; a.D = D; a.F = F; a.act = act; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_mlp_sharded(a, false);
  if (st) return st;
  Plan plan;
  plan_mlp_sharded(a, nullptr, plan);
  keep_plan_text(plan, "mlp_block_sharded");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_mlp_block_sharded(const void* const* X_parts, const void* const* W1t_parts, const void* b1,
                             const void* const* W2t_parts, const void* b2, void* const* Y_parts, int64_t T,
                             int64_t D, int64_t F, int out_dtype, int act, int R_batch, int R_model, void* ws,
                             size_t ws_bytes, void* stream) {
  MlpShardedArgs a;
  a.X = X_parts; a.W1t = W1t_parts; a.b1 = b1; a.W2t = W2t_parts; a.b2 = b2; a.Y = Y_parts;
  a.T = T; a.D = D; a.F = F; a.out = out_dtype; a.act = act; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_mlp_sharded(a, true);
  if (st) return st;
  Plan probe;
  plan_mlp_sharded(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_mlp_sharded(a, ws, plan);
  keep_plan_text(plan, "mlp_block_sharded");
  return execute(plan, stream);
}

// ---- attn_block ------------------------------------------------------------------
size_t partir_attn_block_workspace(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                                   int R_batch, int R_model) {
  AttnArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, B, S, D, n_heads, d_head, 1, 0.f,
             PARTIR_BF16, PARTIR_F32, R_batch, R_model};
  if (validate_attn(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_attn(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_attn_block(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                           int R_batch, int R_model, partir_plan_info* info) {
  AttnArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, B, S, D, n_heads, d_head, 1, 0.f,
             PARTIR_BF16, PARTIR_F32, R_batch, R_model};
  int st = validate_attn(a, false);
  if (st) return st;
  Plan plan;
  plan_attn(a, nullptr, plan);
  keep_plan_text(plan, "attn_block");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_attn_block(const void* X, const void* Wq, const void* Wk, const void* Wv, const void* Wo, void* Y,
                      int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head, int causal, float scale,
                      int in_dtype, int out_dtype, int R_batch, int R_model, void* ws, size_t ws_bytes, void* stream) {
  AttnArgs a{X, Wq, Wk, Wv, Wo, Y, B, S, D, n_heads, d_head, causal ? 1 : 0, scale,
             in_dtype, out_dtype, R_batch, R_model};
  int st = validate_attn(a, true);
  if (st) return st;
  Plan probe;
  plan_attn(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_attn(a, ws, plan);
  keep_plan_text(plan, "attn_block");
  return execute(plan, stream);
}

size_t partir_attn_block_saved_bytes(int64_t B, int64_t S, int64_t D, int64_t n_heads) {
  if (B < 0 || S < 0 || D < 0 || n_heads < 0) return (size_t)-1;
  return attn_core_bytes(B * S, D) + align_up((size_t)(B * S * n_heads) * 4);
}

int partir_attn_block_train(const void* X, const void* Wq, const void* Wk, const void* Wv, const void* Wo,
                            void* Y, void* saved, int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                            int causal, float scale, int in_dtype, int out_dtype, int R_batch, int R_model,
                            void* ws, size_t ws_bytes, void* stream) {
  AttnArgs a{X, Wq, Wk, Wv, Wo, Y, B, S, D, n_heads, d_head, causal ? 1 : 0, scale,
             in_dtype, out_dtype, R_batch, R_model, saved};
  int st = validate_attn(a, true);
  if (st) return st;
  if (B * S > 0 && !saved) return fail(PARTIR_E_NULL, "saved must be non-NULL");
  if (!aligned16(saved)) return fail(PARTIR_E_LAYOUT, "saved must be 16-byte aligned");
  Plan probe;
  plan_attn(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_attn(a, ws, plan);
  keep_plan_text(plan, "attn_block_train");
  return execute(plan, stream);
}

size_t partir_attn_block_backward_workspace(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                                            int R_batch, int R_model) {
  AttnBlockBwdArgs a;
  a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.Rb = R_batch; a.Rm = R_model;
  if (validate_attn_block_bwd(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_attn_block_bwd(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_attn_block_backward(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head, int causal,
                                    int R_batch, int R_model, partir_plan_info* info) {
  AttnBlockBwdArgs a;
  a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.causal = causal ? 1 : 0; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_attn_block_bwd(a, false);
  if (st) return st;
  Plan plan;
  plan_attn_block_bwd(a, nullptr, plan);
  keep_plan_text(plan, "attn_block_backward");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_attn_block_backward(const void* X, const void* Wq, const void* Wk, const void* Wv,
                               const void* Wo, const void* saved, const void* dY, void* dX, void* dWq,
                               void* dWk, void* dWv, void* dWo, int64_t B, int64_t S, int64_t D,
                               int64_t n_heads, int64_t d_head, int causal, float scale, int R_batch, int R_model,
                               void* ws, size_t ws_bytes, void* stream) {
  AttnBlockBwdArgs a;
  a.X = X; a.Wq = Wq; a.Wk = Wk; a.Wv = Wv; a.Wo = Wo; a.saved = saved; a.dY = dY;
  a.dX = dX; a.dWq = dWq; a.dWk = dWk; a.dWv = dWv; a.dWo = dWo;
  a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.causal = causal ? 1 : 0; a.scale = scale;
  a.Rb = R_batch; a.Rm = R_model;
  int st = validate_attn_block_bwd(a, true);
  if (st) return st;
  Plan probe;
  plan_attn_block_bwd(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_attn_block_bwd(a, ws, plan);
  keep_plan_text(plan, "attn_block_backward");
  return execute(plan, stream);
}

// ---- MLP block backward -----------------------------------------------------------
size_t partir_mlp_block_backward_workspace(int64_t T, int64_t D, int64_t F, int act, int with_bias_grads,
                                           int R_batch, int R_model) {
  MlpBwdArgs a;
  a.T = T; a.D = D; a.F = F; a.act = act; a.Rb = R_batch; a.Rm = R_model;
  static char dummy[16] __attribute__((aligned(16)));
  if (with_bias_grads) { a.db1 = dummy; a.db2 = dummy; }
  if (validate_mlp_bwd(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_mlp_bwd(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_mlp_block_backward(int64_t T, int64_t D, int64_t F, int act, int R_batch, int R_model,
                                   partir_plan_info* info) {
  MlpBwdArgs a;
  a.T = T; a.D = D; a.F = F; a.act = act; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_mlp_bwd(a, false);
  if (st) return st;
  Plan plan;
  plan_mlp_bwd(a, nullptr, plan);
  keep_plan_text(plan, "mlp_block_backward");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_mlp_block_backward(const void* X, const void* W1, const void* b1, const void* W2, const void* dY,
                              const void* Z, void* dX, void* dW1, void* db1, void* dW2, void* db2, int64_t T,
                              int64_t D, int64_t F, int act, int R_batch, int R_model, void* ws, size_t ws_bytes,
                              void* stream) {
  MlpBwdArgs a;
  a.X = X; a.W1 = W1; a.b1 = b1; a.W2 = W2; a.dY = dY; a.Z = Z;
  a.dX = dX; a.dW1 = dW1; a.db1 = db1; a.dW2 = dW2; a.db2 = db2;
  a.T = T; a.D = D; a.F = F; a.act = act; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_mlp_bwd(a, true);
  if (st) return st;
  Plan probe;
  plan_mlp_bwd(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_mlp_bwd(a, ws, plan);
  keep_plan_text(plan, "mlp_block_backward");
  return execute(plan, stream);
}

// ---- attention core ---------------------------------------------------------------
size_t partir_attention_workspace(int64_t B, int64_t S, int64_t n_heads, int64_t d_head, int R_kv) {
  AttnCoreArgs a{nullptr, nullptr, nullptr, nullptr, B, S, n_heads, d_head, 1, 0.f, R_kv};
  if (validate_attn_core(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_attn_core(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_attention(int64_t B, int64_t S, int64_t n_heads, int64_t d_head, int causal, int R_kv,
                          partir_plan_info* info) {
  AttnCoreArgs a{nullptr, nullptr, nullptr, nullptr, B, S, n_heads, d_head, causal ? 1 : 0, 0.f, R_kv};
  int st = validate_attn_core(a, false);
  if (st) return st;
  Plan plan;
  plan_attn_core(a, nullptr, plan);
  keep_plan_text(plan, "attention");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_attention(const void* Q, const void* K, const void* V, void* O, int64_t B, int64_t S,
                     int64_t n_heads, int64_t d_head, int causal, float scale, int R_kv, void* ws,
                     size_t ws_bytes, void* stream) {
  AttnCoreArgs a{Q, K, V, O, B, S, n_heads, d_head, causal ? 1 : 0, scale, R_kv};
  int st = validate_attn_core(a, true);
  if (st) return st;
  Plan probe;
  plan_attn_core(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_attn_core(a, ws, plan);
  keep_plan_text(plan, "attention");
  return execute(plan, stream);
}

int partir_attention_train(const void* Q, const void* K, const void* V, void* O, float* lse, int64_t B, int64_t S,
                           int64_t n_heads, int64_t d_head, int causal, float scale, int R_kv, void* ws,
                           size_t ws_bytes, void* stream) {
  AttnCoreArgs a{Q, K, V, O, B, S, n_heads, d_head, causal ? 1 : 0, scale, R_kv, lse};
  int st = validate_attn_core(a, true);
  if (st) return st;
  if (B * S > 0 && !lse) return fail(PARTIR_E_NULL, "lse must be non-NULL");
  if ((uintptr_t)lse & 3) return fail(PARTIR_E_LAYOUT, "lse must be 4-byte aligned");
  Plan probe;
  plan_attn_core(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_attn_core(a, ws, plan);
  keep_plan_text(plan, "attention_train");
  return execute(plan, stream);
}

size_t partir_attention_backward_workspace(int64_t B, int64_t S, int64_t n_heads, int64_t d_head) {
  AttnBwdArgs a;
  a.B = B; a.S = S; a.H = n_heads; a.dh = d_head;
  if (validate_attn_bwd(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_attn_bwd(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_attention_backward(int64_t B, int64_t S, int64_t n_heads, int64_t d_head, int causal,
                                   partir_plan_info* info) {
  AttnBwdArgs a;
  a.B = B; a.S = S; a.H = n_heads; a.dh = d_head; a.causal = causal ? 1 : 0;
  int st = validate_attn_bwd(a, false);
  if (st) return st;
  Plan plan;
  plan_attn_bwd(a, nullptr, plan);
  keep_plan_text(plan, "attention_backward");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_attention_backward(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                              const float* lse, void* dQ, void* dK, void* dV, int64_t B, int64_t S, int64_t n_heads,
                              int64_t d_head, int causal, float scale, void* ws, size_t ws_bytes, void* stream) {
  AttnBwdArgs a;
  a.Q = Q; a.K = K; a.V = V; a.O = O; a.dO = dO; a.lse = lse; a.dQ = dQ; a.dK = dK; a.dV = dV;
  a.B = B; a.S = S; a.H = n_heads; a.dh = d_head; a.causal = causal ? 1 : 0; a.scale = scale;
  int st = validate_attn_bwd(a, true);
  if (st) return st;
  Plan probe;
  plan_attn_bwd(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_attn_bwd(a, ws, plan);
  keep_plan_text(plan, "attention_backward");
  return execute(plan, stream);
}

// ---- decoder_layer ---------------------------------------------------------------
size_t partir_decoder_layer_workspace(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                                      int64_t F, int R_batch, int R_model) {
  DecArgs a;
  a.eps = 1e-6f; a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.F = F; a.Rb = R_batch; a.Rm = R_model;
  if (validate_dec(a, false) != PARTIR_OK) return (size_t)-1;
  Plan plan;
  plan_dec(a, nullptr, plan);
  return plan.ws_bytes;
}

int partir_plan_decoder_layer(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head, int64_t F,
                              int R_batch, int R_model, partir_plan_info* info) {
  DecArgs a;
  a.eps = 1e-6f; a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.F = F; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_dec(a, false);
  if (st) return st;
  Plan plan;
  plan_dec(a, nullptr, plan);
  keep_plan_text(plan, "decoder_layer");
  fill_info(plan, info);
  return PARTIR_OK;
}

int partir_decoder_layer(void* x, const void* g1, const void* g2, float eps, const void* Wq, const void* Wk,
                         const void* Wv, const void* Wo, const void* W1, const void* W2, int64_t B, int64_t S,
                         int64_t D, int64_t n_heads, int64_t d_head, int64_t F, int R_batch, int R_model,
                         void* ws, size_t ws_bytes, void* stream) {
  DecArgs a;
  a.x = x; a.g1 = g1; a.g2 = g2; a.Wq = Wq; a.Wk = Wk; a.Wv = Wv; a.Wo = Wo; a.W1 = W1; a.W2 = W2;
  a.eps = eps; a.B = B; a.S = S; a.D = D; a.H = n_heads; a.dh = d_head; a.F = F; a.Rb = R_batch; a.Rm = R_model;
  int st = validate_dec(a, true);
  if (st) return st;
  Plan probe;
  plan_dec(a, nullptr, probe);
  if ((st = check_ws(probe, ws, ws_bytes))) return st;
  Plan plan;
  plan_dec(a, ws, plan);
  keep_plan_text(plan, "decoder_layer");
  return execute(plan, stream);
}

// ---- trace ------------------------------------------------------------------------
int partir_trace_enable(int on) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  g_trace_on = on != 0;
  return PARTIR_OK;
}

void partir_trace_reset(void) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  for (auto& r : g_trace_pending) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_trace_pending.clear();
  g_trace_totals.clear();
}

int partir_trace_read(partir_trace_entry* out, int max) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  for (auto& r : g_trace_pending) {
    if (hipEventSynchronize(r.stop) != hipSuccess) return -fail(PARTIR_E_HIP, "hipEventSynchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) return -fail(PARTIR_E_HIP, "hipEventElapsedTime failed");
    auto& t = g_trace_totals[r.name];
    t.first += 1;
    t.second += ms;
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_trace_pending.clear();
  int i = 0;
  for (auto& kv : g_trace_totals) {
    if (out && i < max) {
      memset(out[i].name, 0, sizeof out[i].name);
      strncpy(out[i].name, kv.first.c_str(), sizeof out[i].name - 1);
      out[i].launches = kv.second.first;
      out[i].total_ms = kv.second.second;
    }
    ++i;
  }
  return i;
}

}  // extern "C"
