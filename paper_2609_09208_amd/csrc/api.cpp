// C ABI of libpotattn (declared in include/pot_attn.h).
//
// Every check runs on the host before any HIP call; a rejected call touches
// neither the device nor the stream. Launches are asynchronous on the
// caller's stream and allocate nothing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "pot_attn.h"
#include "pot_device.hpp"
#include "pot_launch.hpp"

using namespace potattn;

namespace {

thread_local std::string g_last_error;

pot_status fail(pot_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

}  // namespace

pot_status potattn::report_error(pot_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

namespace {

pot_status ok() {
  g_last_error.clear();
  return POT_OK;
}

pot_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(POT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

constexpr int kE = 6;
constexpr int kMaxF = 12;

pot_status check_format(const pot_format* f) {
  if (!f) return fail(POT_ERR_INVALID_ARG, "fmt is NULL");
  if (f->head_dim != 64) return fail(POT_ERR_UNSUPPORTED, "head_dim %d (only 64)", f->head_dim);
  if (f->exp_bits != 3) return fail(POT_ERR_UNSUPPORTED, "exp_bits %d (only 3)", f->exp_bits);
  if (f->mant_bits < 0 || f->mant_bits > 4)
    return fail(POT_ERR_UNSUPPORTED, "mant_bits %d (0..4)", f->mant_bits);
  if (f->frac_bits < kE)
    return fail(POT_ERR_INVALID_ARG,
                "frac_bits %d < E = %d: a shift F - e would be a right shift", f->frac_bits, kE);
  if (f->frac_bits > kMaxF)
    return fail(POT_ERR_UNSUPPORTED, "frac_bits %d > %d (int32 head-room)", f->frac_bits, kMaxF);
  if (f->hadamard != 0 && f->hadamard != 1)
    return fail(POT_ERR_INVALID_ARG, "hadamard %d (0 or 1)", f->hadamard);
  return POT_OK;
}

struct Plan {
  int n_splits, split_len;
};

// Key splits: enough workgroups to fill the GPU's resident slots in a single
// dispatch round (slots = CUs x resident workgroups per CU); one split when
// the (batch, kv head) pairs alone fill it. Splits are whole 256-key tiles.
Plan plan_from_count(int T, int S) {
  const int tiles = (T + kTile - 1) / kTile;
  S = std::max(1, std::min(S, tiles));
  const int tiles_per_split = (tiles + S - 1) / S;
  Plan p;
  p.split_len = tiles_per_split * kTile;
  p.n_splits = (T + p.split_len - 1) / p.split_len;
  return p;
}

int split_count_for_slots(long units, long slots) {
  return units >= slots ? 1 : (int)(slots / units);
}

// Split count when the grid would fill the GPU's resident slots with short
// splits: splits of at least two 256-key tiles, unless that leaves fewer
// than 256 workgroups (one per CU) when the keys allow more. Measured with
// the four-wave split combine: B = 1, T = 32768: 18.6 us with 64 two-tile
// splits, 19.2 us with 128 one-tile splits, 22.5 us with 32 four-tile
// splits; B = 1, T = 4096: 17.1 us with 16 one-tile splits, 17.5 us with 8.
constexpr int kMinTilesPerSplit = 2;
constexpr long kMinWorkgroups = 256;

int split_count_short_ranges(long units, int tiles) {
  const int s_len = std::max(1, tiles / kMinTilesPerSplit);
  const int s_spread = (int)std::min<long>(tiles, (kMinWorkgroups + units - 1) / units);
  return std::max(s_len, s_spread);
}

// Upper bound used to size workspaces without a device query: 256 CUs x 8
// resident workgroups (the decode kernels reach at most 4 per CU: 4 waves per SIMD).
constexpr long kMaxSlots = 256L * 8;

Plan plan_bound(int B, int Hkv, int T) {
  return plan_from_count(T, split_count_for_slots((long)B * Hkv, kMaxSlots));
}

std::atomic<int> g_cus[64];
// [default / CU-wide variant][score mode][value format][G][mant_bits]
std::atomic<int> g_occ[2][4][3][9][5];

int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  int cus = g_cus[dev].load(std::memory_order_relaxed);
  if (cus <= 0) {
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    g_cus[dev].store(cus, std::memory_order_relaxed);
  }
  return cus;
}

long device_slots(int mode, int G, int mant_bits, int vf, bool pool) {
  const int cus = device_cus();
  std::atomic<int>& slot = g_occ[pool ? 1 : 0][mode][vf][G][mant_bits];
  int occ = slot.load(std::memory_order_relaxed);
  if (occ <= 0) {
    occ = decode_occupancy(mode, G, mant_bits, vf, pool);
    if (occ <= 0) occ = pool ? 1 : 2;
    slot.store(occ, std::memory_order_relaxed);
  }
  return (long)cus * occ;
}

// The CU-wide variant (one workgroup of pool_waves(...) waves per CU, tiles
// claimed from a shared counter) replaces the four-wave workgroups when its
// plan still gives every CU a workgroup and every wave two tiles on average.
constexpr int kPoolTilesPerWave = 2;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct WsLayout {
  size_t qbuf, part_m, part_l, part_o, total;
};

// Workspace: one slot of prepared query operands per decode workgroup
// (B * Hkv * S slots; each workgroup writes its own and reads it back through
// the scalar cache), then the split partials.
WsLayout ws_layout(long B, long Hq, long Hkv, long S) {
  WsLayout w;
  w.qbuf = 0;
  w.part_m = align_up((size_t)(B * Hkv * S) * query_words((int)(Hq / Hkv)) * 4, 256);
  w.part_l = w.part_m + align_up((size_t)(B * Hq * S) * 4, 256);
  w.part_o = w.part_l + align_up((size_t)(B * Hq * S) * 4, 256);
  w.total = w.part_o + align_up((size_t)(B * Hq * S) * 64 * 4, 256);
  return w;
}

bool shape_ok(int B, int Hq, int Hkv, int T) {
  return B >= 1 && Hq >= 1 && Hkv >= 1 && T >= 1 && Hq % Hkv == 0;
}

// Validates the GQA head map and fills DecodeArgs::q_of_kv ([Hkv][G]).
pot_status check_heads(const int32_t* map, int Hq, int Hkv, DecodeArgs* a, int* G_out) {
  if (!map) return fail(POT_ERR_INVALID_ARG, "kv_head_of_q is NULL");
  if (Hq > kMaxHqArg) return fail(POT_ERR_UNSUPPORTED, "Hq %d > %d", Hq, kMaxHqArg);
  if (Hq % Hkv) return fail(POT_ERR_UNSUPPORTED, "Hq %d not a multiple of Hkv %d", Hq, Hkv);
  const int G = Hq / Hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(POT_ERR_UNSUPPORTED, "group size %d (1, 2, 4 or 8)", G);
  std::vector<int> fill(Hkv, 0);
  for (int i = 0; i < Hq; ++i) {
    const int h = map[i];
    if (h < 0 || h >= Hkv)
      return fail(POT_ERR_INVALID_ARG, "kv_head_of_q[%d] = %d outside [0, %d)", i, h, Hkv);
    if (fill[h] >= G)
      return fail(POT_ERR_UNSUPPORTED, "kv head %d serves more than %d query heads", h, G);
    a->q_of_kv[h * G + fill[h]++] = i;
  }
  *G_out = G;
  return POT_OK;
}

// Shared tail of the three decode entry points.
pot_status decode_common(int mode, int mant_bits, DecodeArgs& a, const int32_t* map, int B,
                         int Hq, int Hkv, int T, int64_t t_cap, void* workspace,
                         size_t ws_bytes, pot_debug* dbg, void* stream, int vf = 0) {
  const bool v8 = vf != 0;
  if (!shape_ok(B, Hq, Hkv, T))
    return fail(POT_ERR_INVALID_ARG, "bad shape B=%d Hq=%d Hkv=%d T=%d", B, Hq, Hkv, T);
  if (t_cap < T) return fail(POT_ERR_INVALID_ARG, "T %d > t_cap %lld", T, (long long)t_cap);
  if (T > kMaxKeys)
    return fail(POT_ERR_UNSUPPORTED, "T %d > %d keys per sequence (32-bit buffer ranges)", T,
                kMaxKeys);
  if (t_cap % 8)
    return fail(POT_ERR_INVALID_ARG, "t_cap %lld is not a multiple of 8 (value-cache groups)",
                (long long)t_cap);
  if (v8) {
    if (!a.q || !a.v8 || !a.v_exp || !a.out)
      return fail(POT_ERR_INVALID_ARG, "q, v_u8, v_exp or out is NULL");
    if (!aligned(a.q, 16) || !aligned(a.v8, 16) || !aligned(a.v_exp, 16) || !aligned(a.out, 16))
      return fail(POT_ERR_INVALID_ARG, "q, v_u8, v_exp and out must be 16-byte aligned");
  } else {
    if (!a.q || !a.v || !a.out) return fail(POT_ERR_INVALID_ARG, "q, v or out is NULL");
    if (!aligned(a.q, 16) || !aligned(a.v, 16) || !aligned(a.out, 16))
      return fail(POT_ERR_INVALID_ARG, "q, v and out must be 16-byte aligned");
  }
  if (!workspace) return fail(POT_ERR_INVALID_ARG, "workspace is NULL");
  if (!aligned(workspace, 256))
    return fail(POT_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  int G = 0;
  pot_status st = check_heads(map, Hq, Hkv, &a, &G);
  if (st != POT_OK) return st;
  const int force = dbg ? dbg->force_splits : 0;
  if (force < 0) return fail(POT_ERR_INVALID_ARG, "force_splits %d < 0", force);
  const int mbits = (mode == kScorePot || mode == kScoreDs4a) ? mant_bits : 0;
  const int pw = pool_waves(mode, mbits, vf);
  const int want = dbg ? dbg->force_wg_waves : 0;
  if (want != 0 && want != kBlock / 64 && (pw == 0 || want != pw))
    return fail(POT_ERR_INVALID_ARG, "force_wg_waves %d is neither 0, %d nor %d", want,
                kBlock / 64, pw);
  const long units = (long)B * Hkv;
  Plan p;
  bool pool = false;
  if (force > 0) {
    p = plan_from_count(T, force);
    pool = pw > 0 && (want == pw || (want == 0 && units * p.n_splits >= device_cus() &&
                                     p.split_len >= kPoolTilesPerWave * pw * 64));
  } else {
    if (pw > 0 && want != kBlock / 64) {
      const int S = split_count_for_slots(units, device_slots(mode, G, mbits, vf, true));
      const Plan pp = plan_from_count(T, std::min(S, plan_bound(B, Hkv, T).n_splits));
      if (want == pw ||
          (units * pp.n_splits >= device_cus() && pp.split_len >= kPoolTilesPerWave * pw * 64)) {
        p = pp;
        pool = true;
      }
    }
    if (!pool) {
      const int S = split_count_for_slots(units, device_slots(mode, G, mbits, vf, false));
      const int tiles = (T + kTile - 1) / kTile;
      const int s_short = split_count_short_ranges(units, tiles);
      p = plan_from_count(T, std::min({S, s_short, plan_bound(B, Hkv, T).n_splits}));
    }
  }
  const WsLayout w = ws_layout(B, Hq, Hkv, p.n_splits);
  if (ws_bytes < w.total)
    return fail(POT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed for %d splits", ws_bytes,
                w.total, p.n_splits);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  a.qbuf = reinterpret_cast<int32_t*>(ws + w.qbuf);
  a.qstride = query_words(G);
  a.part_m = reinterpret_cast<int32_t*>(ws + w.part_m);
  a.part_l = reinterpret_cast<float*>(ws + w.part_l);
  a.part_o = reinterpret_cast<float*>(ws + w.part_o);
  a.t_cap = t_cap;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.T = T;
  a.n_splits = p.n_splits;
  a.split_len = p.split_len;
  a.wg_waves = pool ? pw : kBlock / 64;
  bool debug = false;
  hipEvent_t ev_begin = nullptr, ev_end = nullptr;
  if (dbg) {
    ev_begin = static_cast<hipEvent_t>(dbg->decode_begin);
    ev_end = static_cast<hipEvent_t>(dbg->decode_end);
    a.dbg_qhat = dbg->qhat;
    a.dbg_delta = dbg->delta;
    a.dbg_scores = dbg->scores;
    a.dbg_m_final = dbg->m_final;
    a.dbg_m_split = dbg->m_split;
    debug = dbg->qhat || dbg->delta || dbg->scores || dbg->m_final || dbg->m_split;
    dbg->n_splits = p.n_splits;
    dbg->split_len = p.split_len;
    dbg->wg_waves = a.wg_waves;
    if (debug && mode == kScoreFp16)
      return fail(POT_ERR_UNSUPPORTED, "debug taps are not available on the fp16 path");
  }
  return hip_status(
      launch_decode(mode, G, mant_bits, debug, vf, a, static_cast<hipStream_t>(stream), ev_begin,
                    ev_end),
      "decode launch");
}

// Shared body of the INT8-value entry points; vf 1: softmax weights, 2:
// power-of-two weights.
pot_status decode_v8(int vf, const pot_format* fmt, int32_t engine, const float* q,
                                   const uint8_t* codes_se, const uint8_t* codes_m,
                                   const float* key_scale, const uint8_t* v_u8,
                                   const int8_t* v_exp, int64_t t_cap,
                                   const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                   int32_t Hkv, int32_t T, float* out, void* workspace,
                                   size_t ws_bytes, pot_debug* dbg, void* stream) {
  pot_status st = check_format(fmt);
  if (st != POT_OK) return st;
  if (engine != 0 && engine != 1)
    return fail(POT_ERR_INVALID_ARG, "engine %d (0 shift-accumulate, 1 byte decode)", engine);
  if (engine == 1 && fmt->mant_bits != 0)
    return fail(POT_ERR_UNSUPPORTED, "the byte-decode path scores PoT-4 codes only (mant_bits 0)");
  if (!codes_se || !key_scale) return fail(POT_ERR_INVALID_ARG, "codes_se or key_scale is NULL");
  if ((fmt->mant_bits > 0) != (codes_m != nullptr))
    return fail(POT_ERR_INVALID_ARG, "codes_m must be non-NULL exactly when mant_bits > 0");
  if (!aligned(codes_se, 16) || !aligned(key_scale, 4) || (codes_m && !aligned(codes_m, 8)))
    return fail(POT_ERR_INVALID_ARG, "misaligned codes_se / key_scale / codes_m");
  DecodeArgs a{};
  a.q = q;
  a.codes_se = codes_se;
  a.codes_m = codes_m;
  a.key_scale = key_scale;
  a.v8 = v_u8;
  a.v_exp = v_exp;
  a.out = out;
  a.frac_bits = fmt->frac_bits;
  a.hadamard = fmt->hadamard;
  return decode_common(engine == 0 ? kScorePot : kScoreDs4a, fmt->mant_bits, a, kv_head_of_q, B,
                       Hq, Hkv, T, t_cap, workspace, ws_bytes, dbg, stream, vf);
}

}  // namespace

extern "C" {

const char* pot_status_string(pot_status s) {
  switch (s) {
    case POT_OK: return "POT_OK";
    case POT_ERR_INVALID_ARG: return "POT_ERR_INVALID_ARG";
    case POT_ERR_UNSUPPORTED: return "POT_ERR_UNSUPPORTED";
    case POT_ERR_WORKSPACE: return "POT_ERR_WORKSPACE";
    case POT_ERR_HIP: return "POT_ERR_HIP";
  }
  return "POT_ERR_UNKNOWN";
}

const char* pot_last_error(void) { return g_last_error.c_str(); }

size_t pot_code_bytes_per_row(const pot_format* fmt) {
  if (check_format(fmt) != POT_OK) return 0;
  return 32 + 8 * (size_t)fmt->mant_bits;
}

pot_status pot_encode_keys(const pot_format* fmt, const uint16_t* k_fp16, int64_t n_rows,
                           int64_t out_row_stride, int32_t scale_mode, float* key_scale,
                           uint8_t* codes_se, uint8_t* codes_m, void* stream) {
  pot_status st = check_format(fmt);
  if (st != POT_OK) return st;
  if (n_rows < 0) return fail(POT_ERR_INVALID_ARG, "n_rows %lld < 0", (long long)n_rows);
  if (out_row_stride < 1)
    return fail(POT_ERR_INVALID_ARG, "out_row_stride %lld < 1", (long long)out_row_stride);
  if (scale_mode != 0 && scale_mode != 1)
    return fail(POT_ERR_INVALID_ARG, "scale_mode %d (0 or 1)", scale_mode);
  if (n_rows == 0) return ok();
  if (!k_fp16 || !key_scale || !codes_se)
    return fail(POT_ERR_INVALID_ARG, "k_fp16, key_scale or codes_se is NULL");
  if ((fmt->mant_bits > 0) != (codes_m != nullptr))
    return fail(POT_ERR_INVALID_ARG, "codes_m must be non-NULL exactly when mant_bits > 0");
  if (!aligned(k_fp16, 16) || !aligned(codes_se, 16) || !aligned(key_scale, 4) ||
      (codes_m && !aligned(codes_m, 8)))
    return fail(POT_ERR_INVALID_ARG, "misaligned k_fp16 / codes_se / key_scale / codes_m");
  if (n_rows > (int64_t)1 << 36) return fail(POT_ERR_INVALID_ARG, "n_rows too large");
  const EncodeTables tab = make_encode_tables(fmt->mant_bits);
  return hip_status(launch_encode_pot(k_fp16, n_rows, out_row_stride, scale_mode, fmt->hadamard,
                                      key_scale, codes_se, codes_m, tab,
                                      static_cast<hipStream_t>(stream)),
                    "encode launch");
}

pot_status pot_store_values(const uint16_t* v_fp16, int64_t n_seq, int64_t n_tok, int64_t t_cap,
                            int64_t t0, uint16_t* v_cache, void* stream) {
  if (n_seq < 0 || n_tok < 0)
    return fail(POT_ERR_INVALID_ARG, "n_seq %lld / n_tok %lld < 0", (long long)n_seq,
                (long long)n_tok);
  if (t_cap < 8 || t_cap % 8)
    return fail(POT_ERR_INVALID_ARG, "t_cap %lld is not a positive multiple of 8",
                (long long)t_cap);
  if (t0 < 0 || t0 + n_tok > t_cap)
    return fail(POT_ERR_INVALID_ARG, "tokens [%lld, %lld) outside [0, t_cap = %lld)",
                (long long)t0, (long long)(t0 + n_tok), (long long)t_cap);
  if (n_seq == 0 || n_tok == 0) return ok();
  if (!v_fp16 || !v_cache) return fail(POT_ERR_INVALID_ARG, "v_fp16 or v_cache is NULL");
  if (!aligned(v_fp16, 16) || !aligned(v_cache, 16))
    return fail(POT_ERR_INVALID_ARG, "v_fp16 and v_cache must be 16-byte aligned");
  return hip_status(launch_store_values(v_fp16, n_seq, n_tok, t_cap, t0, v_cache,
                                        static_cast<hipStream_t>(stream)),
                    "store values launch");
}

pot_status pot_store_values_int8(const uint16_t* v_fp16, int64_t n_seq, int64_t n_tok,
                                 int64_t t_cap, int64_t t0, uint8_t* v_u8, int8_t* v_exp,
                                 void* stream) {
  if (n_seq < 0 || n_tok < 0)
    return fail(POT_ERR_INVALID_ARG, "n_seq %lld / n_tok %lld < 0", (long long)n_seq,
                (long long)n_tok);
  if (t_cap < 8 || t_cap % 8)
    return fail(POT_ERR_INVALID_ARG, "t_cap %lld is not a positive multiple of 8",
                (long long)t_cap);
  if (t0 < 0 || t0 + n_tok > t_cap)
    return fail(POT_ERR_INVALID_ARG, "tokens [%lld, %lld) outside [0, t_cap = %lld)",
                (long long)t0, (long long)(t0 + n_tok), (long long)t_cap);
  if (n_seq == 0 || n_tok == 0) return ok();
  if (!v_fp16 || !v_u8 || !v_exp)
    return fail(POT_ERR_INVALID_ARG, "v_fp16, v_u8 or v_exp is NULL");
  if (!aligned(v_fp16, 16) || !aligned(v_u8, 16) || !aligned(v_exp, 16))
    return fail(POT_ERR_INVALID_ARG, "v_fp16, v_u8 and v_exp must be 16-byte aligned");
  if (n_seq > ((int64_t)1 << 31) / n_tok)
    return fail(POT_ERR_INVALID_ARG, "n_seq * n_tok too large");
  return hip_status(launch_store_values_i8(v_fp16, n_seq, n_tok, t_cap, t0, v_u8, v_exp,
                                           static_cast<hipStream_t>(stream)),
                    "store values launch");
}

size_t pot_decode_workspace_bytes(int32_t B, int32_t Hq, int32_t Hkv, int32_t T) {
  if (!shape_ok(B, Hq, Hkv, T)) return 0;
  return ws_layout(B, Hq, Hkv, plan_bound(B, Hkv, T).n_splits).total;
}

size_t pot_decode_workspace_bytes_for_splits(int32_t B, int32_t Hq, int32_t Hkv, int32_t T,
                                             int32_t n_splits) {
  if (!shape_ok(B, Hq, Hkv, T) || n_splits < 0) return 0;
  const Plan p = n_splits > 0 ? plan_from_count(T, n_splits) : plan_bound(B, Hkv, T);
  return ws_layout(B, Hq, Hkv, p.n_splits).total;
}

pot_status pot_workspace_init(void* workspace, size_t ws_bytes, void* stream) {
  if (!workspace) return fail(POT_ERR_INVALID_ARG, "workspace is NULL");
  return hip_status(launch_fill_zero(workspace, ws_bytes, static_cast<hipStream_t>(stream)),
                    "workspace init");
}

pot_status pot_decode_attention(const pot_format* fmt, const float* q, const uint8_t* codes_se,
                                const uint8_t* codes_m, const float* key_scale,
                                const uint16_t* v_cache, int64_t t_cap,
                                const int32_t* kv_head_of_q, int32_t B, int32_t Hq, int32_t Hkv,
                                int32_t T, float* out, void* workspace, size_t ws_bytes,
                                pot_debug* dbg, void* stream) {
  pot_status st = check_format(fmt);
  if (st != POT_OK) return st;
  if (!codes_se || !key_scale) return fail(POT_ERR_INVALID_ARG, "codes_se or key_scale is NULL");
  if ((fmt->mant_bits > 0) != (codes_m != nullptr))
    return fail(POT_ERR_INVALID_ARG, "codes_m must be non-NULL exactly when mant_bits > 0");
  if (!aligned(codes_se, 16) || !aligned(key_scale, 4) || (codes_m && !aligned(codes_m, 8)))
    return fail(POT_ERR_INVALID_ARG, "misaligned codes_se / key_scale / codes_m");
  DecodeArgs a{};
  a.q = q;
  a.codes_se = codes_se;
  a.codes_m = codes_m;
  a.key_scale = key_scale;
  a.v = v_cache;
  a.out = out;
  a.frac_bits = fmt->frac_bits;
  a.hadamard = fmt->hadamard;
  return decode_common(kScorePot, fmt->mant_bits, a, kv_head_of_q, B, Hq, Hkv, T, t_cap,
                       workspace, ws_bytes, dbg, stream);
}

pot_status pot_append_decode_attention(const pot_format* fmt, const float* q,
                                       const uint16_t* k_new, const uint16_t* v_new,
                                       uint8_t* codes_se, uint8_t* codes_m, float* key_scale,
                                       uint16_t* v_cache, int64_t t_cap,
                                       const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                       int32_t Hkv, int32_t T, float* out, void* workspace,
                                       size_t ws_bytes, pot_debug* dbg, void* stream) {
  pot_status st = check_format(fmt);
  if (st != POT_OK) return st;
  if (!k_new || !v_new) return fail(POT_ERR_INVALID_ARG, "k_new or v_new is NULL");
  if (!aligned(k_new, 16) || !aligned(v_new, 16))
    return fail(POT_ERR_INVALID_ARG, "k_new and v_new must be 16-byte aligned");
  if (!codes_se || !key_scale) return fail(POT_ERR_INVALID_ARG, "codes_se or key_scale is NULL");
  if ((fmt->mant_bits > 0) != (codes_m != nullptr))
    return fail(POT_ERR_INVALID_ARG, "codes_m must be non-NULL exactly when mant_bits > 0");
  if (!aligned(codes_se, 16) || !aligned(key_scale, 4) || (codes_m && !aligned(codes_m, 8)))
    return fail(POT_ERR_INVALID_ARG, "misaligned codes_se / key_scale / codes_m");
  DecodeArgs a{};
  a.q = q;
  a.codes_se = codes_se;
  a.codes_m = codes_m;
  a.key_scale = key_scale;
  a.v = v_cache;
  a.out = out;
  a.frac_bits = fmt->frac_bits;
  a.hadamard = fmt->hadamard;
  a.app_k = k_new;
  a.app_v = v_new;
  a.app_codes_se = codes_se;
  a.app_codes_m = codes_m;
  a.app_key_scale = key_scale;
  a.app_v_cache = v_cache;
  a.app_tab = make_encode_tables(fmt->mant_bits);
  return decode_common(kScorePot, fmt->mant_bits, a, kv_head_of_q, B, Hq, Hkv, T, t_cap,
                       workspace, ws_bytes, dbg, stream);
}

pot_status pot_decode_attention_v8(const pot_format* fmt, int32_t engine, const float* q,
                                   const uint8_t* codes_se, const uint8_t* codes_m,
                                   const float* key_scale, const uint8_t* v_u8,
                                   const int8_t* v_exp, int64_t t_cap,
                                   const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                   int32_t Hkv, int32_t T, float* out, void* workspace,
                                   size_t ws_bytes, pot_debug* dbg, void* stream) {
  return decode_v8(1, fmt, engine, q, codes_se, codes_m, key_scale, v_u8, v_exp, t_cap,
                   kv_head_of_q, B, Hq, Hkv, T, out, workspace, ws_bytes, dbg, stream);
}

pot_status pot_decode_attention_v8_pow2(const pot_format* fmt, int32_t engine, const float* q,
                                        const uint8_t* codes_se, const uint8_t* codes_m,
                                        const float* key_scale, const uint8_t* v_u8,
                                        const int8_t* v_exp, int64_t t_cap,
                                        const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                        int32_t Hkv, int32_t T, float* out, void* workspace,
                                        size_t ws_bytes, pot_debug* dbg, void* stream) {
  return decode_v8(2, fmt, engine, q, codes_se, codes_m, key_scale, v_u8, v_exp, t_cap,
                   kv_head_of_q, B, Hq, Hkv, T, out, workspace, ws_bytes, dbg, stream);
}

pot_status pot_append_decode_attention_v8(const pot_format* fmt, int32_t engine,
                                          const float* q, const uint16_t* k_new,
                                          const uint16_t* v_new, uint8_t* codes_se,
                                          uint8_t* codes_m, float* key_scale, uint8_t* v_u8,
                                          int8_t* v_exp, int64_t t_cap,
                                          const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                          int32_t Hkv, int32_t T, float* out, void* workspace,
                                          size_t ws_bytes, pot_debug* dbg, void* stream) {
  pot_status st = check_format(fmt);
  if (st != POT_OK) return st;
  if (engine != 0 && engine != 1)
    return fail(POT_ERR_INVALID_ARG, "engine %d (0 shift-accumulate, 1 byte decode)", engine);
  if (engine == 1 && fmt->mant_bits != 0)
    return fail(POT_ERR_UNSUPPORTED, "the byte-decode path scores PoT-4 codes only (mant_bits 0)");
  if (!k_new || !v_new) return fail(POT_ERR_INVALID_ARG, "k_new or v_new is NULL");
  if (!aligned(k_new, 16) || !aligned(v_new, 16))
    return fail(POT_ERR_INVALID_ARG, "k_new and v_new must be 16-byte aligned");
  if (!codes_se || !key_scale) return fail(POT_ERR_INVALID_ARG, "codes_se or key_scale is NULL");
  if ((fmt->mant_bits > 0) != (codes_m != nullptr))
    return fail(POT_ERR_INVALID_ARG, "codes_m must be non-NULL exactly when mant_bits > 0");
  if (!aligned(codes_se, 16) || !aligned(key_scale, 4) || (codes_m && !aligned(codes_m, 8)))
    return fail(POT_ERR_INVALID_ARG, "misaligned codes_se / key_scale / codes_m");
  DecodeArgs a{};
  a.q = q;
  a.codes_se = codes_se;
  a.codes_m = codes_m;
  a.key_scale = key_scale;
  a.v8 = v_u8;
  a.v_exp = v_exp;
  a.out = out;
  a.frac_bits = fmt->frac_bits;
  a.hadamard = fmt->hadamard;
  a.app_k = k_new;
  a.app_v = v_new;
  a.app_codes_se = codes_se;
  a.app_codes_m = codes_m;
  a.app_key_scale = key_scale;
  a.app_v8 = v_u8;
  a.app_v_exp = v_exp;
  a.app_tab = make_encode_tables(fmt->mant_bits);
  return decode_common(engine == 0 ? kScorePot : kScoreDs4a, fmt->mant_bits, a, kv_head_of_q, B,
                       Hq, Hkv, T, t_cap, workspace, ws_bytes, dbg, stream, 1);
}

pot_status pot_ds4a_decode_attention(const pot_format* fmt, const float* q,
                                     const uint8_t* codes_se, const float* key_scale,
                                     const uint16_t* v_cache, int64_t t_cap,
                                     const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                     int32_t Hkv, int32_t T, float* out, void* workspace,
                                     size_t ws_bytes, pot_debug* dbg, void* stream) {
  pot_status st = check_format(fmt);
  if (st != POT_OK) return st;
  if (fmt->mant_bits != 0)
    return fail(POT_ERR_UNSUPPORTED, "the byte-decode path scores PoT-4 codes only (mant_bits 0)");
  if (!codes_se || !key_scale) return fail(POT_ERR_INVALID_ARG, "codes_se or key_scale is NULL");
  if (!aligned(codes_se, 16) || !aligned(key_scale, 4))
    return fail(POT_ERR_INVALID_ARG, "misaligned codes_se / key_scale");
  DecodeArgs a{};
  a.q = q;
  a.codes_se = codes_se;
  a.key_scale = key_scale;
  a.v = v_cache;
  a.out = out;
  a.frac_bits = fmt->frac_bits;
  a.hadamard = fmt->hadamard;
  return decode_common(kScoreDs4a, 0, a, kv_head_of_q, B, Hq, Hkv, T, t_cap, workspace, ws_bytes,
                       dbg, stream);
}

pot_status pot_dot_decode_attention(const pot_format* fmt, const float* q,
                                    const uint8_t* codes_se, const uint8_t* codes_m,
                                    const float* key_scale, const uint16_t* v_cache,
                                    int64_t t_cap, const int32_t* kv_head_of_q, int32_t B,
                                    int32_t Hq, int32_t Hkv, int32_t T, float* out,
                                    void* workspace, size_t ws_bytes, pot_debug* dbg,
                                    void* stream) {
  pot_status st = check_format(fmt);
  if (st != POT_OK) return st;
  if (!codes_se || !key_scale) return fail(POT_ERR_INVALID_ARG, "codes_se or key_scale is NULL");
  if ((fmt->mant_bits > 0) != (codes_m != nullptr))
    return fail(POT_ERR_INVALID_ARG, "codes_m must be non-NULL exactly when mant_bits > 0");
  if (!aligned(codes_se, 16) || !aligned(key_scale, 4) || (codes_m && !aligned(codes_m, 8)))
    return fail(POT_ERR_INVALID_ARG, "misaligned codes_se / key_scale / codes_m");
  DecodeArgs a{};
  a.q = q;
  a.codes_se = codes_se;
  a.codes_m = codes_m;
  a.key_scale = key_scale;
  a.v = v_cache;
  a.out = out;
  a.frac_bits = fmt->frac_bits;
  a.hadamard = fmt->hadamard;
  return decode_common(kScoreDs4a, fmt->mant_bits, a, kv_head_of_q, B, Hq, Hkv, T, t_cap,
                       workspace, ws_bytes, dbg, stream);
}

pot_status pot_int8_encode_keys(const uint16_t* k_fp16, int64_t n_rows, int64_t out_row_stride,
                                int32_t hadamard, float* key_scale, int8_t* codes, void* stream) {
  if (n_rows < 0) return fail(POT_ERR_INVALID_ARG, "n_rows %lld < 0", (long long)n_rows);
  if (out_row_stride < 1)
    return fail(POT_ERR_INVALID_ARG, "out_row_stride %lld < 1", (long long)out_row_stride);
  if (hadamard != 0 && hadamard != 1)
    return fail(POT_ERR_INVALID_ARG, "hadamard %d (0 or 1)", hadamard);
  if (n_rows == 0) return ok();
  if (!k_fp16 || !key_scale || !codes)
    return fail(POT_ERR_INVALID_ARG, "k_fp16, key_scale or codes is NULL");
  if (!aligned(k_fp16, 16) || !aligned(codes, 16) || !aligned(key_scale, 4))
    return fail(POT_ERR_INVALID_ARG, "misaligned k_fp16 / codes / key_scale");
  return hip_status(launch_encode_int8(k_fp16, n_rows, out_row_stride, hadamard, key_scale,
                                       codes, static_cast<hipStream_t>(stream)),
                    "int8 encode launch");
}

pot_status pot_int8_decode_attention(const float* q, const int8_t* codes, const float* key_scale,
                                     const uint16_t* v_cache, int64_t t_cap,
                                     const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                     int32_t Hkv, int32_t T, int32_t hadamard, float* out,
                                     void* workspace, size_t ws_bytes, pot_debug* dbg,
                                     void* stream) {
  if (hadamard != 0 && hadamard != 1)
    return fail(POT_ERR_INVALID_ARG, "hadamard %d (0 or 1)", hadamard);
  if (!codes || !key_scale) return fail(POT_ERR_INVALID_ARG, "codes or key_scale is NULL");
  if (!aligned(codes, 16) || !aligned(key_scale, 4))
    return fail(POT_ERR_INVALID_ARG, "misaligned codes / key_scale");
  DecodeArgs a{};
  a.q = q;
  a.codes_i8 = codes;
  a.key_scale = key_scale;
  a.v = v_cache;
  a.out = out;
  a.hadamard = hadamard;
  return decode_common(kScoreInt8, 0, a, kv_head_of_q, B, Hq, Hkv, T, t_cap, workspace, ws_bytes,
                       dbg, stream);
}

pot_status pot_fp16_decode_attention(const float* q, const uint16_t* k_fp16,
                                     const uint16_t* v_cache, int64_t t_cap,
                                     const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                     int32_t Hkv, int32_t T, float* out, void* workspace,
                                     size_t ws_bytes, void* stream) {
  if (!k_fp16) return fail(POT_ERR_INVALID_ARG, "k_fp16 is NULL");
  if (!aligned(k_fp16, 16)) return fail(POT_ERR_INVALID_ARG, "k_fp16 must be 16-byte aligned");
  DecodeArgs a{};
  a.q = q;
  a.k_f16 = k_fp16;
  a.v = v_cache;
  a.out = out;
  return decode_common(kScoreFp16, 0, a, kv_head_of_q, B, Hq, Hkv, T, t_cap, workspace, ws_bytes,
                       nullptr, stream);
}

}  // extern "C"
