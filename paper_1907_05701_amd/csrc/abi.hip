// Host-side plumbing of the C ABI: dims validation, the flat parameter layout
// (PyTorch nn.LSTM order, as the paper trains with PyTorch, Section 5.1),
// workspace layout, error strings and the optional kernel-timing hooks.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <string>
#include <vector>

#include "common.hpp"
#include "gemm.hpp"
#include "lstm_persist.hpp"

static thread_local char g_err[512] = "";

int blstm_fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int blstm_check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return blstm_fail(BLSTM_EHIP, "%s: %s", what, hipGetErrorString(e));
  return BLSTM_OK;
}

extern "C" const char* blstm_last_error(void) { return g_err; }

// Split-K factor of a product with Mo x No outputs (per batch) and Kr-long
// reductions: enough workgroups to cover the chip, at least 4 k-tiles per
// split, below 256 tiles.  bf16 (direct-to-LDS kernel) aims at 256
// workgroups (measured: more splits cost more in the partial reduction than
// they gain), float32 at 512.
int plan_splits(int64_t Mo, int64_t No, int64_t Kr, int BMt, int BNt, int BK, int batches, bool lp, bool alone) {
  const int64_t tiles = cdiv(Mo, BMt) * cdiv(No, BNt) * batches;
  if (tiles >= 256) return 1;
  // a product launched alone (bf16) fills one round of two blocks per CU
  // without starting a second; the backward layer products share a grouped
  // launch and split to half a round each
  int64_t s = lp && alone ? std::max<int64_t>(512 / tiles, 1) : cdiv(lp ? 256 : 512, tiles);
  const int64_t kt = cdiv(Kr, BK);
  s = std::min<int64_t>(s, std::max<int64_t>(kt / 4, 1));
  s = std::min<int64_t>(s, 16);
  return (int)std::max<int64_t>(s, 1);
}

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

int make_layout(const blstm_dims* d, Layout* lo) {
  if (!d || !lo) return blstm_fail(BLSTM_EINVAL, "null dims");
  if (d->L < 1 || d->D < 1 || d->H < 1 || d->P < 1 || d->K < 1 || d->T < 1 || d->B < 1)
    return blstm_fail(BLSTM_EINVAL, "all dims must be positive (L=%d D=%d H=%d P=%d K=%d T=%d B=%d)",
                      d->L, d->D, d->H, d->P, d->K, d->T, d->B);
  if (d->precision != BLSTM_FP32 && d->precision != BLSTM_BF16)
    return blstm_fail(BLSTM_EINVAL, "precision must be BLSTM_FP32 or BLSTM_BF16");
  if (d->L > MAX_LAYERS) return blstm_fail(BLSTM_EUNSUPPORTED, "L > %d", MAX_LAYERS);
  const int hq = d->precision == BLSTM_BF16 ? 32 : 16;
  if (d->H % hq) return blstm_fail(BLSTM_EUNSUPPORTED, "H must be a multiple of %d", hq);
  if (d->P % 8) return blstm_fail(BLSTM_EUNSUPPORTED, "P must be a multiple of 8");
  if (d->D % 4) return blstm_fail(BLSTM_EUNSUPPORTED, "D must be a multiple of 4");
  if ((int64_t)d->T * d->B > (1 << 24)) return blstm_fail(BLSTM_EUNSUPPORTED, "T*B too large");
  if (d->B > 65535 * 16) return blstm_fail(BLSTM_EUNSUPPORTED, "B too large");

  Layout& L = *lo;
  memset(&L, 0, sizeof(L));
  L.L = d->L; L.D = d->D; L.H = d->H; L.P = d->P; L.K = d->K; L.T = d->T; L.B = d->B;
  L.prec = d->precision;
  L.M = (int64_t)d->T * d->B;
  L.Dp0 = (int)rup(d->D, 8);
  L.Kp = (int)rup(d->K, 8);
  L.es = d->precision == BLSTM_BF16 ? 2 : 4;
  const int64_t H = d->H;
  int64_t off = 0;
  for (int l = 0; l < d->L; ++l) {
    const int64_t Dl = l == 0 ? d->D : 2 * H;
    for (int dir = 0; dir < 2; ++dir) {
      L.Wih[l][dir] = off; off += 4 * H * Dl;
      L.Whh[l][dir] = off; off += 4 * H * H;
      L.bih[l][dir] = off; off += 4 * H;
      L.bhh[l][dir] = off; off += 4 * H;
    }
  }
  L.Wl = off; off += (int64_t)d->P * 2 * H;
  L.bl = off; off += d->P;
  L.Ws = off; off += (int64_t)d->K * d->P;
  L.bs = off; off += d->K;
  L.n = off;

  // act_ws
  const size_t es = L.es;
  const int64_t M = L.M;
  size_t a = 0;
  L.X0 = a; a = align256(a + (size_t)M * L.Dp0 * es);
  for (int l = 0; l < d->L; ++l) {
    if (l < d->L - 1) { L.Y[l] = a; a = align256(a + (size_t)M * 2 * H * es); }
    L.G[l] = a; a = align256(a + (size_t)M * 8 * H * es);
    L.C[l] = a; a = align256(a + (size_t)M * 2 * H * 4);
  }
  L.GX = a; a = align256(a + (size_t)M * 8 * H * es);
  L.DYa = a; a = align256(a + (size_t)M * 2 * H * 4);
  L.DYb = a; a = align256(a + (size_t)M * 2 * H * 4);
  L.DC = a; a = align256(a + (size_t)2 * d->B * H * 4);
  L.WT = a; a = align256(a + (size_t)2 * d->L * 4 * H * H * es);
  L.WP0_bytes = es == 2 && d->D % 8 != 0 ? (size_t)2 * 4 * H * L.Dp0 * es : 0;
  L.WP0 = a; a = align256(a + L.WP0_bytes);
  // bf16 with B % 8 == 0: the BPTT kernels also write da frame-contiguous
  // (da^T), the A operand of the weight gradients
  L.write_dat = es == 2 && d->B % 8 == 0;
  // da^T [8H][M], one per layer (the weight gradients of every layer run
  // after the last BPTT; the side-stream path alternates two of them)
  L.dat_bytes = align256(L.write_dat ? (size_t)M * 8 * H * es : 0);
  L.DAT = a; a += (size_t)std::max(2, d->L) * L.dat_bytes;
  // per-step 16-row partials (per-step BPTT) or per-workgroup partials over
  // all steps (persistent BPTT, 8-row workgroups)
  L.dbp_bytes = align256((size_t)std::max<int64_t>((int64_t)d->T * cdiv(d->B, 16), cdiv(d->B, 8)) * 8 * H * 4);
  L.DBP = a; a += (size_t)std::max(2, d->L) * L.dbp_bytes;   // per layer when the bias sums wait for the last BPTT
  L.CSP = a; a = align256(a + (size_t)COLSUM_MAX_CHUNKS * 8 * H * 4);
  // split-K plans and partial buffers of the backward GEMMs
  const int BMt = es == 2 ? GemmCfg<bf16>::BM : GemmCfg<float>::BM;
  const int BNt = es == 2 ? GemmCfg<bf16>::BN : GemmCfg<float>::BN;
  const int BKt = es == 2 ? GemmCfg<bf16>::BK : GemmCfg<float>::BK;
  // each layer's three products own disjoint partial regions (dW_ih, dW_hh,
  // dX), so that they can run as one grouped launch.  bf16, measured on
  // MI355X at the learner-step shapes: dX splits to fill one round of two
  // blocks per CU by itself and dW_hh is not split (its partial pass costs
  // more than the parallelism gains: 1.207 -> 1.253 M frames/s); dW_ih keeps
  // half a round.  A sweep of the other products' splits and of the tile
  // order's row grouping found the defaults at the optimum.
  size_t skp = 0;
  const bool lp = es == 2;
  for (int l = 0; l < d->L; ++l) {
    const int64_t Dl = l == 0 ? d->D : 2 * H;
    const bool with_dx = l > 0;
    L.sp_dWih[l] = plan_splits(4 * H, Dl, M, BMt, BNt, BKt, 2, lp, false);
    const size_t ih_bytes = L.sp_dWih[l] > 1 ? align256((size_t)L.sp_dWih[l] * 2 * 4 * H * Dl * 4) : 0;
    L.sp_dWhh[l] = lp ? 1 : plan_splits(4 * H, H, (int64_t)(d->T - 1) * d->B, BMt, BNt, BKt, 2, lp, false);
    const size_t hh_bytes = L.sp_dWhh[l] > 1 ? align256((size_t)L.sp_dWhh[l] * 2 * 4 * H * H * 4) : 0;
    L.sp_dX[l] = with_dx ? plan_splits(M, Dl, 8 * H, BMt, BNt, BKt, 1, lp, lp) : 1;
    const size_t dx_bytes = L.sp_dX[l] > 1 ? align256((size_t)L.sp_dX[l] * M * Dl * 4) : 0;
    L.skp_hh[l] = ih_bytes;
    L.skp_dx[l] = ih_bytes + hh_bytes;
    skp = std::max(skp, ih_bytes + hh_bytes + dx_bytes);
  }
  L.SKP = a; a = align256(a + skp);
  L.SKP2 = a; a = align256(a + skp);   // split-K partials of the side-stream products
  L.XCH = a; a = align256(a + persist_xch_bytes(d->B, d->H));   // recurrent step exchange
  // recurrence status block, the last PERSIST_STATUS_BYTES of act_ws
  L.SYNC = a; a += PERSIST_STATUS_BYTES;
  L.act_bytes = a;

  // head_ws
  size_t h = 0;
  const int64_t P = d->P;
  L.Z = h; h = align256(h + (size_t)M * P * es);
  // float32: the logits, overwritten by ds; bf16: ds only (the logits stay
  // in the products' accumulators) plus the per-(frame, class strip)
  // statistics and the per-frame log-sum-exp
  L.S = h; h = align256(h + (size_t)M * L.Kp * es);
  L.LST = h; h = align256(h + (es == 2 ? (size_t)M * cdiv(d->K, 64) * 8 : 0));
  L.LSE = h; h = align256(h + (es == 2 ? (size_t)M * 4 : 0));
  L.LDB = h; h = align256(h + (es == 2 ? (size_t)cdiv(M, 32) * L.Kp * 4 : 0));   // db_s partials per frame tile (32 frames or more)
  // bf16: db_l shares of the 128-class strips (W_s^T db_s, per strip)
  L.DBLP = h; h = align256(h + (es == 2 ? (size_t)cdiv(d->K, 128) * d->P * 4 : 0));
  L.RL = h; h = align256(h + (size_t)M * 4);
  L.DZ = h; h = align256(h + (size_t)M * P * 4);
  L.DZT = h; h = align256(h + (size_t)M * P * es);
  // column-sum partials: db_l (P columns), and db_s on the float32 path
  L.HCSP = h; h = align256(h + (size_t)COLSUM_MAX_CHUNKS * (es == 2 ? P : std::max<int64_t>(L.Kp, P)) * 4);
  size_t hsk = 0;
  L.sp_z = es == 2 ? plan_splits(M, P, 2 * H, BMt, BNt, BKt, 1, true, true) : 1;
  if (L.sp_z > 1) hsk = std::max(hsk, (size_t)L.sp_z * M * P * 4);
  L.sp_dz = plan_splits(M, P, d->K, BMt, BNt, BKt, 1, es == 2, true);
  hsk = std::max(hsk, (size_t)L.sp_dz * M * P * 4);  // dz always goes through partials
  L.sp_dWs = plan_splits(d->K, P, M, BMt, BNt, BKt, 1, es == 2, true);
  if (L.sp_dWs > 1) hsk = std::max(hsk, (size_t)L.sp_dWs * d->K * P * 4);
  L.sp_dWl = plan_splits(P, 2 * H, M, BMt, BNt, BKt, 1, es == 2, true);
  if (L.sp_dWl > 1) hsk = std::max(hsk, (size_t)L.sp_dWl * P * 2 * H * 4);
  L.sp_dy = plan_splits(M, 2 * H, P, BMt, BNt, BKt, 1, es == 2, true);
  if (L.sp_dy > 1) hsk = std::max(hsk, (size_t)L.sp_dy * M * 2 * H * 4);
  L.HSKP = h; h = align256(h + hsk);
  L.head_bytes = h;
  L.ytop_bytes = (size_t)M * 2 * H * es;
  return BLSTM_OK;
}

extern "C" int64_t blstm_param_count(const blstm_dims* dims) {
  Layout lo;
  int rc = make_layout(dims, &lo);
  if (rc != BLSTM_OK) return rc;
  return lo.n;
}

extern "C" int blstm_workspace_bytes(const blstm_dims* dims, size_t* act_ws, size_t* head_ws,
                                     size_t* theta_lp, size_t* y_top) {
  Layout lo;
  int rc = make_layout(dims, &lo);
  if (rc != BLSTM_OK) return rc;
  if (act_ws) *act_ws = lo.act_bytes;
  if (head_ws) *head_ws = lo.head_bytes;
  if (theta_lp) *theta_lp = lo.prec == BLSTM_BF16 ? (size_t)lo.n * 2 : 0;
  if (y_top) *y_top = lo.ytop_bytes;
  return BLSTM_OK;
}

// ---------------------------------------------------------------------------
// Kernel timing: HIP events around selected launches.
// ---------------------------------------------------------------------------
bool g_timing_on = false;
static std::string g_prefix;
struct TimedLaunch {
  std::string name;
  hipEvent_t start, stop;
  int launches;
};
static std::vector<TimedLaunch> g_launches;
static std::vector<hipEvent_t> g_pool;

static hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

int timing_pre(const char* name, hipStream_t s) { return timing_pre_n(name, s, 1); }

int timing_pre_n(const char* name, hipStream_t s, int launches) {
  if (strncmp(name, g_prefix.c_str(), g_prefix.size()) != 0) return -1;
  TimedLaunch t;
  t.name = name;
  t.launches = launches;
  t.start = take_event();
  t.stop = take_event();
  if (!t.start || !t.stop) return -1;
  hipEventRecord(t.start, s);
  g_launches.push_back(t);
  return (int)g_launches.size() - 1;
}

void timing_post(int slot, hipStream_t s) { hipEventRecord(g_launches[slot].stop, s); }

extern "C" int blstm_timing_begin(const char* prefix) {
  for (auto& t : g_launches) {
    g_pool.push_back(t.start);
    g_pool.push_back(t.stop);
  }
  g_launches.clear();
  g_prefix = prefix ? prefix : "";
  g_timing_on = true;
  return BLSTM_OK;
}

extern "C" int blstm_timing_end(blstm_kernel_time* out, int32_t cap, int32_t* count) {
  g_timing_on = false;
  std::vector<blstm_kernel_time> agg;
  for (auto& t : g_launches) {
    if (hipEventSynchronize(t.stop) != hipSuccess)
      return blstm_fail(BLSTM_EHIP, "hipEventSynchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.start, t.stop) != hipSuccess)
      return blstm_fail(BLSTM_EHIP, "hipEventElapsedTime failed");
    size_t i = 0;
    for (; i < agg.size(); ++i)
      if (t.name == agg[i].name) break;
    if (i == agg.size()) {
      blstm_kernel_time k;
      memset(&k, 0, sizeof(k));
      snprintf(k.name, sizeof(k.name), "%s", t.name.c_str());
      agg.push_back(k);
    }
    agg[i].launches += t.launches;
    agg[i].total_ms += ms;
  }
  if (count) *count = (int32_t)agg.size();
  for (size_t i = 0; i < agg.size() && (int32_t)i < cap; ++i) out[i] = agg[i];
  return BLSTM_OK;
}
