// C ABI of the KV-rebuild library: argument validation, wave planning,
// metadata staging and the per-layer kernel sequence of the rebuild and of the
// resumed decode step.  Host code only; the kernels live in misc.hip,
// gemm_bf16.hip, gemm_f32.hip, attention.hip and decode.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <set>
#include <string>
#include <vector>

#include "kvr.h"
#include "kvr_decode.h"
#include "kvr_verify.h"
#include "kvr_reuse.h"
#include "kvr_profile.h"
#include "launch.h"

using namespace kvr;

namespace {

thread_local std::string g_err;

kv_status fail(kv_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

kv_status ok() {
  g_err.clear();
  return KV_OK;
}

}  // namespace

// error reporting for the other host files of the library (ipc.hip)
namespace kvr_err {
kv_status set(kv_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}
kv_status clear() { return ok(); }
}  // namespace kvr_err

namespace {

int64_t elem_bytes(int32_t dtype) { return dtype == KV_BF16 ? 2 : 4; }
int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

kv_status check_desc(const kv_model_desc* d) {
  if (!d) return fail(KV_EINVAL, "null model description");
  if (d->num_layers <= 0 || d->hidden <= 0 || d->num_q_heads <= 0 || d->num_kv_heads <= 0 ||
      d->head_dim <= 0 || d->ffn_dim <= 0 || d->vocab <= 0)
    return fail(KV_EINVAL, "model dimensions must be positive");
  if (!(d->rms_eps >= 0.0) || !(d->rope_theta > 0.0))
    return fail(KV_EINVAL, "rms_eps must be >= 0 and rope_theta > 0");
  if (d->num_q_heads % d->num_kv_heads != 0)
    return fail(KV_EINVAL, "num_q_heads must be a multiple of num_kv_heads");
  if (d->hidden % 8 != 0 || d->hidden > 8192)
    return fail(KV_EINVAL, "hidden must be a multiple of 8 and at most 8192");
  if ((d->qk_norm != 0 && d->qk_norm != 1) || (d->qkv_bias != 0 && d->qkv_bias != 1))
    return fail(KV_EINVAL, "qk_norm and qkv_bias must be 0 or 1");
  if (d->qk_norm && d->head_dim < 32) return fail(KV_EINVAL, "qk_norm needs head_dim >= 32");
  if (d->dtype == KV_BF16) {
    if (d->head_dim != 128) return fail(KV_EINVAL, "bf16 models need head_dim == 128");
    if (d->hidden % 256 != 0) return fail(KV_EINVAL, "bf16 models need hidden % 256 == 0");
    if (d->num_kv_heads % 2 != 0) return fail(KV_EINVAL, "bf16 models need an even num_kv_heads");
    if (d->ffn_dim % 128 != 0) return fail(KV_EINVAL, "bf16 models need ffn_dim % 128 == 0");
  } else if (d->dtype == KV_F32) {
    if (d->head_dim % 2 != 0 || 128 % d->head_dim != 0 || d->head_dim < 16)
      return fail(KV_EINVAL, "fp32 models need head_dim in {16, 32, 64, 128}");
    if ((d->num_kv_heads * d->head_dim) % 128 != 0 || (d->num_q_heads * d->head_dim) % 128 != 0)
      return fail(KV_EINVAL, "fp32 models need nq*d and nkv*d multiples of 128");
    if (d->hidden % 128 != 0) return fail(KV_EINVAL, "fp32 models need hidden % 128 == 0");
    if (d->ffn_dim % 8 != 0) return fail(KV_EINVAL, "fp32 models need ffn_dim % 8 == 0");
  } else {
    return fail(KV_EINVAL, "unknown dtype %d", d->dtype);
  }
  return KV_OK;
}

bool same_desc(const kv_model_desc& a, const kv_model_desc& b) {
  return a.num_layers == b.num_layers && a.hidden == b.hidden && a.num_q_heads == b.num_q_heads &&
         a.num_kv_heads == b.num_kv_heads && a.head_dim == b.head_dim && a.ffn_dim == b.ffn_dim &&
         a.vocab == b.vocab && a.rms_eps == b.rms_eps && a.rope_theta == b.rope_theta &&
         a.dtype == b.dtype && a.qk_norm == b.qk_norm && a.qkv_bias == b.qkv_bias;
}

// ---------------------------------------------------------------------------
// Workspace layout (256-byte aligned segments; metadata first so that one
// host->device copy stages it)
// ---------------------------------------------------------------------------
struct Layout {
  int64_t Tg = 0, W = 0, Wpad = 0, Tk = 0, Wk = 0, Wkpad = 0, nqblk_cap = 0, nseg_cap = 0;
  size_t tok = 0, pos = 0, slot = 0, krow = 0, kslot = 0, qblk = 0, seg = 0, meta_end = 0;
  size_t rope = 0, x = 0, a = 0, q = 0, u = 0, vt = 0, kc = 0, hf = 0, total = 0;
};

// Two row spaces.  Rows (Tg in all, W per wave) are the positions computed:
// each request occupies round_up(len - start, ROW_ALIGN) of them.  Key rows
// (Tk, Wk) hold the K/V copies attention reads: round_up(start + its rows,
// ROW_ALIGN) per request, the retained prefix first.  With every start 0 the
// two spaces coincide.  nseg_cap bounds the prefix-gather segments.
Layout make_layout(const kv_model_desc& d, int32_t R, int64_t Tg, int64_t W, int64_t Tk, int64_t Wk,
                   int64_t nseg_cap) {
  Layout L;
  L.Tg = Tg;
  L.W = W;
  L.Wpad = round_up(std::max<int64_t>(W, 1), 256);
  L.Tk = Tk;
  L.Wk = Wk;
  L.Wkpad = round_up(std::max<int64_t>(Wk, 1), 256);
  L.nqblk_cap = (Tg + ATTN_QBLOCK_MIN - 1) / ATTN_QBLOCK_MIN + R;
  L.nseg_cap = nseg_cap;
  const int64_t e = elem_bytes(d.dtype);
  size_t off = 0;
  auto seg = [&](size_t bytes) {
    const size_t at = off;
    off = (size_t)round_up((int64_t)(off + bytes), 256);
    return at;
  };
  L.tok = seg(4 * (size_t)Tg);
  L.pos = seg(4 * (size_t)Tg);
  L.slot = seg(8 * (size_t)Tg);
  L.krow = seg(4 * (size_t)Tg);
  L.kslot = seg(8 * (size_t)Tk);
  L.qblk = seg(16 * (size_t)L.nqblk_cap);
  L.seg = seg(8 * (size_t)nseg_cap);
  L.meta_end = off;
  L.rope = seg((size_t)8 * L.Wkpad * (d.head_dim / 2));
  L.x = seg((size_t)4 * L.Wpad * d.hidden);
  L.a = seg((size_t)e * L.Wpad * d.hidden);
  L.q = seg((size_t)e * L.Wpad * d.num_q_heads * d.head_dim);
  L.u = seg((size_t)e * L.Wpad * d.num_q_heads * d.head_dim);
  L.vt = seg(d.dtype == KV_BF16 ? (size_t)2 * d.num_kv_heads * d.head_dim * L.Wkpad : 0);
  L.kc = seg(d.dtype == KV_BF16 ? (size_t)2 * d.num_kv_heads * d.head_dim * L.Wkpad : 0);
  L.hf = seg((size_t)e * L.Wpad * d.ffn_dim);
  L.total = off;
  return L;
}

// ---------------------------------------------------------------------------
// Handles
// ---------------------------------------------------------------------------
int64_t padded_rows(int64_t n) { return n > 0 ? round_up(n, ROW_ALIGN) : 0; }

// Key rows a wave gets for a row capacity W: the rows' share of all key
// rows, at least the largest request's key rows.
int64_t key_capacity(int64_t W, int64_t Tg, int64_t Tk, int64_t kmax) {
  if (Tg <= 0) return kmax;
  const int64_t prop = round_up((W * Tk + Tg - 1) / Tg, ROW_ALIGN);
  return std::max(kmax, std::min(Tk, prop));
}

struct Wave {
  int64_t tok_begin;  // first row of the wave
  int32_t rows;       // rows including per-request padding (a multiple of ROW_ALIGN)
  int64_t key_begin;  // first key row of the wave
  int32_t keys;       // key rows
  int32_t qblk_begin, num_qblk;
  int32_t seg_begin, num_seg;
  double causal_pairs;  // (query, key) pairs of its computed positions
  int64_t tokens;       // real (unpadded) computed positions
};

}  // namespace

struct kv_arena {
  void* base;
  uint64_t bytes;
  kv_model_desc desc;
  int32_t block_size;
  int64_t num_blocks;
  int32_t device;
  int* probe_flag;
  // pinned host staging for metadata uploads; reused after its last copy completed
  void* pinned = nullptr;
  size_t pinned_bytes = 0;
  hipEvent_t staged = nullptr;
  bool staged_pending = false;
  // optional per-kernel-class timing
  bool profile = false;
  std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> prof_pending;
  std::vector<hipEvent_t> prof_pool;
  double prof_ms[KV_PROF_CLASSES] = {};
  int64_t prof_launches[KV_PROF_CLASSES] = {};
  double prof_flops[KV_PROF_CLASSES] = {};
  std::vector<double> pending_flops;
};

struct kv_plan {
  kv_arena* arena;
  char* ws;
  uint64_t ws_bytes;
  Layout lay;
  std::vector<Wave> waves;
  int32_t max_len;   // longest request with positions to compute
  bool has_prefix;   // some request starts past position 0
};

namespace {

std::mutex g_reg_mu;
std::set<const void*> g_arenas, g_plans;

bool live_arena(const kv_arena* a) {
  std::lock_guard<std::mutex> g(g_reg_mu);
  return a && g_arenas.count(a);
}
bool live_plan(const kv_plan* p) {
  std::lock_guard<std::mutex> g(g_reg_mu);
  return p && g_plans.count(p);
}

struct DeviceGuard {
  int prev = -1;
  bool changed = false;
  hipError_t err = hipSuccess;
  explicit DeviceGuard(int dev) {
    err = hipGetDevice(&prev);
    if (err == hipSuccess && prev != dev) {
      err = hipSetDevice(dev);
      changed = err == hipSuccess;
    }
  }
  ~DeviceGuard() {
    if (changed) (void)hipSetDevice(prev);
  }
};

// starts may be null (every request from position 0).  Rules for starts:
// 0 <= start <= len, start a multiple of 8 unless equal to len.  Blocks:
// a block holding a position >= start of its request is written and may be
// listed by no other request for writing, nor read as prefix by an earlier
// request; a block holding only positions < start is read and may be shared,
// also with an earlier request that writes it.
kv_status check_request(const kv_model_desc* desc, int32_t B, int64_t NB, const int32_t* tokens,
                        const int32_t* lens, int32_t R, const int32_t* tables, int32_t max_blocks,
                        int64_t* total_out, int32_t* max_len_out, const int32_t* starts = nullptr) {
  kv_status st = check_desc(desc);
  if (st != KV_OK) return st;
  if (B <= 0 || NB <= 0) return fail(KV_EINVAL, "block_size and num_blocks must be positive");
  if (R < 0) return fail(KV_EINVAL, "num_requests < 0");
  if (max_blocks < 0) return fail(KV_EINVAL, "max_blocks_per_req < 0");
  if (R > 0 && !lens) return fail(KV_EINVAL, "null prefix_lens");
  int64_t T = 0;
  int32_t max_len = 0;
  for (int32_t r = 0; r < R; ++r) {
    if (lens[r] < 0) return fail(KV_EINVAL, "prefix_lens[%d] = %d < 0", r, lens[r]);
    const int32_t s0 = starts ? starts[r] : 0;
    if (s0 < 0 || s0 > lens[r])
      return fail(KV_EINVAL, "starts[%d] = %d outside [0, %d]", r, s0, lens[r]);
    if (s0 % 8 != 0 && s0 != lens[r])
      return fail(KV_EINVAL, "starts[%d] = %d is not a multiple of 8", r, s0);
    T += lens[r] - s0;
    max_len = std::max(max_len, lens[r]);
  }
  if (T > (int64_t)INT32_MAX) return fail(KV_EINVAL, "more than 2^31-1 prefix tokens in one call");
  if (T > 0 && !tokens) return fail(KV_EINVAL, "null token_prefixes");
  if ((T > 0 || (starts && max_len > 0)) && !tables) return fail(KV_EINVAL, "null block_tables");
  for (int32_t r = 0; r < R; ++r) {
    const int64_t nb = ((int64_t)lens[r] + B - 1) / B;
    if (nb > max_blocks)
      return fail(KV_ECAPACITY, "request %d needs %lld blocks > max_blocks_per_req %d", r,
                  (long long)nb, max_blocks);
  }
  for (int64_t i = 0; i < T; ++i)
    if (tokens[i] < 0 || tokens[i] >= desc->vocab)
      return fail(KV_ERANGE, "token %d at index %lld outside [0, %d)", tokens[i], (long long)i,
                  desc->vocab);
  // writer of each block (-1: none)
  std::vector<int32_t> writer((size_t)NB, -1);
  for (int32_t r = 0; r < R; ++r) {
    const int64_t nb = ((int64_t)lens[r] + B - 1) / B;
    const int64_t s0 = starts ? starts[r] : 0;
    for (int64_t b = 0; b < nb; ++b) {
      const int32_t blk = tables[(int64_t)r * max_blocks + b];
      if (blk < 0 || blk >= NB)
        return fail(KV_ERANGE, "block_tables[%d][%lld] = %d outside [0, %lld)", r, (long long)b,
                    blk, (long long)NB);
      if ((b + 1) * B > s0 && s0 < lens[r]) {  // holds a position >= start: written
        if (writer[blk] >= 0) return fail(KV_EALIAS, "block %d listed twice", blk);
        writer[blk] = r;
      }
    }
  }
  if (starts)
    for (int32_t r = 0; r < R; ++r) {
      const int64_t s0 = starts[r];
      for (int64_t b = 0; b * B < s0; ++b) {  // holds a position < start: read
        const int32_t blk = tables[(int64_t)r * max_blocks + b];
        if (writer[blk] > r)
          return fail(KV_EALIAS, "block %d is read by request %d before request %d writes it", blk, r,
                      writer[blk]);
      }
    }
  if (total_out) *total_out = T;
  if (max_len_out) *max_len_out = max_len;
  return KV_OK;
}

// Decode-step workspace: metadata first (one host->device copy), then the
// per-request activations.  Block tables are staged up to the blocks a step
// uses (at most max_position entries per request, the block size being 1 at
// worst).  The final-norm rows are padded to a multiple of 256: they are the
// B operand of the LM-head GEMM, whose output is the transposed logits
// [vocab][npad].
struct DecodeLayout {
  int32_t R = 0, npad = 0, splits = 0;
  int64_t max_position = 0;
  size_t tok = 0, pos = 0, rowidx = 0, slot = 0, ctx = 0, tables = 0, meta_end = 0;
  size_t rope = 0, x = 0, a = 0, q = 0, u = 0, hf = 0, part = 0, gpart = 0, amax = 0, logit = 0;
  size_t total = 0;
  int64_t gpart_elems = 0;
};

DecodeLayout make_decode_layout(const kv_model_desc& d, int32_t R, int64_t max_position) {
  DecodeLayout L;
  L.R = R;
  L.max_position = max_position;
  L.npad = (int32_t)round_up(std::max<int32_t>(R, 1), 256);
  // split counts shrink as the batch grows: size for one request's
  L.splits = decode_attn_splits(1, d.num_kv_heads, max_position);
  if (d.dtype == KV_BF16) {
    const int H = d.hidden, qd = d.num_q_heads * d.head_dim, kvd = d.num_kv_heads * d.head_dim;
    L.gpart_elems = std::max(
        std::max(gemm_bf16_splitk_part_elems(R, qd + 2 * kvd, H), gemm_bf16_splitk_part_elems(R, H, qd)),
        std::max(gemm_bf16_splitk_part_elems(R, 2 * d.ffn_dim, H),
                 gemm_bf16_splitk_part_elems(R, H, d.ffn_dim)));
  }
  const int64_t e = elem_bytes(d.dtype);
  size_t off = 0;
  auto seg = [&](size_t bytes) {
    const size_t at = off;
    off = (size_t)round_up((int64_t)(off + bytes), 256);
    return at;
  };
  L.tok = seg(4 * (size_t)R);
  L.pos = seg(4 * (size_t)R);
  L.rowidx = seg(4 * (size_t)R);
  L.slot = seg(8 * (size_t)R);
  L.ctx = seg(4 * (size_t)R);
  L.tables = seg(4 * (size_t)R * (size_t)max_position);
  L.meta_end = off;
  L.rope = seg((size_t)8 * R * (d.head_dim / 2));
  L.x = seg((size_t)4 * R * d.hidden);
  L.a = seg((size_t)e * L.npad * d.hidden);
  L.q = seg((size_t)e * R * d.num_q_heads * d.head_dim);
  L.u = seg((size_t)e * R * d.num_q_heads * d.head_dim);
  L.hf = seg((size_t)e * R * d.ffn_dim);
  L.part = seg((size_t)4 * R * d.num_q_heads * L.splits * (d.head_dim + 2));
  L.gpart = seg((size_t)4 * L.gpart_elems);
  L.amax = seg((size_t)8 * ARGMAX_CHUNKS * R);
  L.logit = seg((size_t)4 * d.vocab * L.npad);
  L.total = off;
  return L;
}

kv_status check_decode(const kv_model_desc* desc, int32_t B, int64_t NB, const int32_t* tokens,
                       const int32_t* positions, int32_t R, const int32_t* tables,
                       int32_t max_blocks, int64_t* max_pos_out) {
  kv_status st = check_desc(desc);
  if (st != KV_OK) return st;
  if (desc->num_q_heads / desc->num_kv_heads > 16 || desc->head_dim > 128)
    return fail(KV_EINVAL, "decode supports at most 16 q heads per kv head and head_dim <= 128");
  if (B <= 0 || NB <= 0) return fail(KV_EINVAL, "block_size and num_blocks must be positive");
  if (R < 0) return fail(KV_EINVAL, "num_requests < 0");
  if (max_blocks < 0) return fail(KV_EINVAL, "max_blocks_per_req < 0");
  if (R > 0 && (!tokens || !positions || !tables))
    return fail(KV_EINVAL, "null tokens, positions or block_tables");
  int64_t max_pos = 0;
  for (int32_t r = 0; r < R; ++r) {
    if (positions[r] < 0) return fail(KV_EINVAL, "positions[%d] = %d < 0", r, positions[r]);
    if (tokens[r] < 0 || tokens[r] >= desc->vocab)
      return fail(KV_ERANGE, "token %d of request %d outside [0, %d)", tokens[r], r, desc->vocab);
    if (positions[r] / B >= max_blocks)
      return fail(KV_ECAPACITY, "position %d of request %d needs block %d >= max_blocks_per_req %d",
                  positions[r], r, positions[r] / B, max_blocks);
    max_pos = std::max<int64_t>(max_pos, positions[r]);
  }
  // The block holding a request's new position is written by the step: it
  // may be listed only there, by that request.  Blocks the step only reads
  // (full prefix blocks, for instance shared by several requests) may be
  // listed any number of times.
  for (int32_t r = 0; r < R; ++r)
    for (int32_t b = 0; b <= positions[r] / B; ++b) {
      const int32_t blk = tables[(int64_t)r * max_blocks + b];
      if (blk < 0 || blk >= NB)
        return fail(KV_ERANGE, "block_tables[%d][%d] = %d outside [0, %lld)", r, b, blk,
                    (long long)NB);
    }
  std::vector<int32_t> writer((size_t)NB, -1);
  for (int32_t r = 0; r < R; ++r) {
    const int32_t blk = tables[(int64_t)r * max_blocks + positions[r] / B];
    if (writer[blk] >= 0)
      return fail(KV_EALIAS, "block %d holds the new positions of requests %d and %d", blk, writer[blk], r);
    writer[blk] = r;
  }
  for (int32_t r = 0; r < R; ++r)
    for (int32_t b = 0; b <= positions[r] / B; ++b) {
      const int32_t blk = tables[(int64_t)r * max_blocks + b];
      if (writer[blk] >= 0 && (writer[blk] != r || b != positions[r] / B))
        return fail(KV_EALIAS, "block %d, written by request %d's step, is also listed by request %d "
                    "(entry %d)", blk, writer[blk], r, b);
    }
  if (max_pos_out) *max_pos_out = max_pos;
  return KV_OK;
}

// timing hooks around each launch when profiling is on
struct ProfScope {
  kv_arena* a;
  hipStream_t s;
  int cls;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  ProfScope(kv_arena* a_, hipStream_t s_, int cls_, double flops) : a(a_), s(s_), cls(cls_) {
    if (!a->profile) return;
    auto take = [&]() {
      hipEvent_t e = nullptr;
      if (!a->prof_pool.empty()) {
        e = a->prof_pool.back();
        a->prof_pool.pop_back();
      } else {
        (void)hipEventCreate(&e);
      }
      return e;
    };
    e0 = take();
    e1 = take();
    (void)hipEventRecord(e0, s);
    a->pending_flops.push_back(flops);
  }
  ~ProfScope() {
    if (!e0) return;
    (void)hipEventRecord(e1, s);
    a->prof_pending.push_back({cls, {e0, e1}});
  }
};

}  // namespace

// ---------------------------------------------------------------------------
// Entry points
// ---------------------------------------------------------------------------
extern "C" {

const char* kv_last_error(void) { return g_err.c_str(); }

uint64_t kv_rebuild_workspace_bytes(const kv_model_desc* desc, int32_t num_requests,
                                    int64_t total_tokens, int64_t wave_tokens) {
  if (check_desc(desc) != KV_OK || num_requests < 0 || total_tokens < 0 || wave_tokens < 0)
    return 0;
  // every request may add up to ROW_ALIGN - 1 padding rows
  const int64_t pad = (int64_t)(ROW_ALIGN - 1) * num_requests;
  const int64_t W = std::min(wave_tokens, total_tokens) + pad;
  return make_layout(*desc, num_requests, total_tokens + pad, W, total_tokens + pad, W, 0).total;
}

uint64_t kv_rebuild_from_workspace_bytes(const kv_model_desc* desc, int32_t num_requests,
                                         int64_t total_rows, int64_t total_keys, int64_t wave_rows) {
  if (check_desc(desc) != KV_OK || num_requests < 0 || total_rows < 0 || total_keys < total_rows ||
      wave_rows < 0)
    return 0;
  const int64_t pad = (int64_t)(ROW_ALIGN - 1) * num_requests;
  const int64_t Tg = total_rows + pad, Tk = total_keys + 2 * pad;
  const int64_t W = std::min(wave_rows, total_rows) + pad;
  // gather segments: the prefixes in pieces of GATHER_KEYS, plus at most
  // one partial piece and one zero-fill segment per request
  const int64_t nseg = (total_keys - total_rows) / GATHER_KEYS + 2 * (int64_t)num_requests + 1;
  return make_layout(*desc, num_requests, Tg, W, Tk, key_capacity(W, Tg, Tk, 0), nseg).total;
}

kv_status kv_rebuild_check(const kv_model_desc* desc, int32_t block_size, int64_t num_blocks,
                           const int32_t* token_prefixes, const int32_t* prefix_lens,
                           int32_t num_requests, const int32_t* block_tables,
                           int32_t max_blocks_per_req) {
  kv_status st = check_request(desc, block_size, num_blocks, token_prefixes, prefix_lens,
                               num_requests, block_tables, max_blocks_per_req, nullptr, nullptr);
  return st == KV_OK ? ok() : st;
}

kv_status kv_arena_bind(void* base, uint64_t bytes, const kv_model_desc* desc, int32_t block_size,
                        int64_t num_blocks, int32_t device, kv_arena_t* out) {
  if (!out) return fail(KV_EINVAL, "null output handle");
  *out = nullptr;
  if (!base) return fail(KV_EINVAL, "null arena base");
  kv_status st = check_desc(desc);
  if (st != KV_OK) return st;
  if (block_size <= 0 || num_blocks <= 0)
    return fail(KV_EINVAL, "block_size and num_blocks must be positive");
  const unsigned __int128 need = (unsigned __int128)desc->num_layers * 2 * (uint64_t)num_blocks *
                                 (uint64_t)block_size * desc->num_kv_heads * desc->head_dim *
                                 elem_bytes(desc->dtype);
  if (need > (unsigned __int128)bytes)
    return fail(KV_EINVAL, "arena of %llu bytes is smaller than its geometry needs",
                (unsigned long long)bytes);
  const char* force = getenv("KVR_DEBUG_FAIL_PROBE");
  if (force && force[0] == '1') return fail(KV_EDEVICE, "health probe failed (forced by KVR_DEBUG_FAIL_PROBE)");

  DeviceGuard dg(device);
  if (dg.err != hipSuccess) return fail(KV_EDEVICE, "cannot select device %d: %s", device, hipGetErrorString(dg.err));
  hipPointerAttribute_t attr;
  hipError_t e = hipPointerGetAttributes(&attr, base);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(KV_EDEVICE, "arena pointer not known to HIP: %s", hipGetErrorString(e));
  }
  if (attr.type != hipMemoryTypeDevice || attr.device != device)
    return fail(KV_EDEVICE, "arena pointer is not device memory on device %d", device);
  // health probe: a kernel round trip on the device (Sec. 4.2 step 2)
  int* flag = nullptr;
  if ((e = hipMalloc(&flag, sizeof(int))) != hipSuccess)
    return fail(KV_EDEVICE, "probe allocation failed: %s", hipGetErrorString(e));
  int host_flag = 0;
  bool good = hipMemset(flag, 0, sizeof(int)) == hipSuccess && launch_probe(flag, nullptr) == 0 &&
              hipMemcpy(&host_flag, flag, sizeof(int), hipMemcpyDeviceToHost) == hipSuccess &&
              host_flag == 0x600D;
  if (!good) {
    (void)hipGetLastError();
    (void)hipFree(flag);
    return fail(KV_EDEVICE, "GPU health probe failed on device %d", device);
  }
  kv_arena* a = new (std::nothrow) kv_arena();
  if (!a) {
    (void)hipFree(flag);
    return fail(KV_ENOMEM, "host allocation failed");
  }
  a->base = base;
  a->bytes = bytes;
  a->desc = *desc;
  a->block_size = block_size;
  a->num_blocks = num_blocks;
  a->device = device;
  a->probe_flag = flag;
  if (hipEventCreateWithFlags(&a->staged, hipEventDisableTiming) != hipSuccess) {
    (void)hipFree(flag);
    delete a;
    return fail(KV_EDEVICE, "event creation failed");
  }
  {
    std::lock_guard<std::mutex> g(g_reg_mu);
    g_arenas.insert(a);
  }
  *out = a;
  return ok();
}

kv_status kv_arena_release(kv_arena_t a) {
  {
    std::lock_guard<std::mutex> g(g_reg_mu);
    if (!a || !g_arenas.count(a)) return fail(KV_ESTATE, "unknown or released arena handle");
    g_arenas.erase(a);
  }
  DeviceGuard dg(a->device);
  if (a->staged_pending) (void)hipEventSynchronize(a->staged);
  if (a->pinned) (void)hipHostFree(a->pinned);
  (void)hipEventDestroy(a->staged);
  for (auto& pe : a->prof_pending) {
    (void)hipEventDestroy(pe.second.first);
    (void)hipEventDestroy(pe.second.second);
  }
  for (auto e : a->prof_pool) (void)hipEventDestroy(e);
  (void)hipFree(a->probe_flag);
  delete a;
  return ok();
}

}  // extern "C"

namespace {

kv_status stage_impl(kv_arena_t arena, const int32_t* tokens, const int32_t* lens,
                     const int32_t* starts, int32_t R, const int32_t* tables, int32_t max_blocks,
                     void* workspace, uint64_t ws_bytes, void* stream, kv_plan_t* out) {
  if (!out) return fail(KV_EINVAL, "null output plan");
  *out = nullptr;
  if (!live_arena(arena)) return fail(KV_ESTATE, "unknown or released arena handle");
  int64_t T = 0;
  int32_t max_len = 0;
  kv_status st = check_request(&arena->desc, arena->block_size, arena->num_blocks, tokens, lens, R,
                               tables, max_blocks, &T, &max_len, starts);
  if (st != KV_OK) return st;
  const kv_model_desc& d = arena->desc;
  kv_plan* plan = new (std::nothrow) kv_plan();
  if (!plan) return fail(KV_ENOMEM, "host allocation failed");
  plan->arena = arena;
  plan->ws = reinterpret_cast<char*>(workspace);
  plan->ws_bytes = ws_bytes;
  plan->max_len = max_len;
  plan->has_prefix = false;
  if (T > 0) {
    if (!workspace) {
      delete plan;
      return fail(KV_EINVAL, "null workspace");
    }
    // rows: each request's computed positions start on a ROW_ALIGN boundary;
    // padding rows carry token 0, position 0 and slot -1 (computed, never
    // scattered).  Key rows: the retained prefix, then the computed rows.
    std::vector<int32_t> st0(R, 0);
    for (int32_t r = 0; r < R; ++r) st0[r] = starts ? starts[r] : 0;
    std::vector<int64_t> tok_off(R + 1, 0), row_off(R + 1, 0), key_off(R + 1, 0);
    int64_t gmax = 0, kmax = 0, nseg = 0;
    for (int32_t r = 0; r < R; ++r) {
      const int64_t n = lens[r] - st0[r];
      const int64_t g = padded_rows(n);
      const int64_t k = n > 0 ? round_up(st0[r] + g, ROW_ALIGN) : 0;
      tok_off[r + 1] = tok_off[r] + n;
      row_off[r + 1] = row_off[r] + g;
      key_off[r + 1] = key_off[r] + k;
      gmax = std::max(gmax, g);
      kmax = std::max(kmax, k);
      if (n > 0 && st0[r] > 0) {
        nseg += (st0[r] + GATHER_KEYS - 1) / GATHER_KEYS + (k > st0[r] + g ? 1 : 0);
        plan->has_prefix = true;
      }
    }
    int32_t max_active = 0;
    for (int32_t r = 0; r < R; ++r)
      if (lens[r] > st0[r]) max_active = std::max(max_active, lens[r]);
    plan->max_len = max_active;
    const int64_t Tg = row_off[R], Tk = key_off[R];
    const Layout smallest = make_layout(d, R, Tg, gmax, Tk, kmax, nseg);
    if (smallest.total > ws_bytes) {
      delete plan;
      return fail(KV_ENOMEM, "workspace of %llu bytes < %llu needed for the longest request",
                  (unsigned long long)ws_bytes, (unsigned long long)smallest.total);
    }
    // largest row capacity whose layout fits
    int64_t lo = gmax, hi = Tg;
    while (lo < hi) {
      const int64_t mid = lo + (hi - lo + 1) / 2;
      if (make_layout(d, R, Tg, mid, Tk, key_capacity(mid, Tg, Tk, kmax), nseg).total <= ws_bytes)
        lo = mid;
      else
        hi = mid - 1;
    }
    plan->lay = make_layout(d, R, Tg, lo, Tk, key_capacity(lo, Tg, Tk, kmax), nseg);
    const Layout& L = plan->lay;

    // waves: consecutive requests, never split, within both capacities
    std::vector<int32_t> wave_of(R, -1);
    {
      Wave w{0, 0, 0, 0, 0, 0, 0, 0, 0.0, 0};
      for (int32_t r = 0; r < R; ++r) {
        const int64_t n = lens[r] - st0[r];
        if (n == 0) continue;
        const int64_t g = row_off[r + 1] - row_off[r], k = key_off[r + 1] - key_off[r];
        if (w.rows > 0 && (w.rows + g > L.W || w.keys + k > L.Wk)) {
          plan->waves.push_back(w);
          w = Wave{row_off[r], 0, key_off[r], 0, 0, 0, 0, 0, 0.0, 0};
        }
        if (w.rows == 0) {
          w.tok_begin = row_off[r];
          w.key_begin = key_off[r];
        }
        w.rows += (int32_t)g;
        w.keys += (int32_t)k;
        const double a = (double)st0[r], b = (double)lens[r];
        w.causal_pairs += 0.5 * (b * (b + 1.0) - a * (a + 1.0));
        w.tokens += n;
        wave_of[r] = (int32_t)plan->waves.size();
      }
      if (w.rows > 0) plan->waves.push_back(w);
    }

    // metadata image in pinned host memory, then one async copy
    if (arena->staged_pending) {
      (void)hipEventSynchronize(arena->staged);
      arena->staged_pending = false;
    }
    DeviceGuard dg(arena->device);
    if (arena->pinned_bytes < L.meta_end) {
      if (arena->pinned) (void)hipHostFree(arena->pinned);
      arena->pinned = nullptr;
      arena->pinned_bytes = 0;
      if (hipHostMalloc(&arena->pinned, L.meta_end, hipHostMallocDefault) != hipSuccess) {
        arena->pinned = nullptr;
        delete plan;
        return fail(KV_ENOMEM, "pinned staging allocation of %zu bytes failed", (size_t)L.meta_end);
      }
      arena->pinned_bytes = L.meta_end;
    }
    char* hb = reinterpret_cast<char*>(arena->pinned);
    int32_t* htok = reinterpret_cast<int32_t*>(hb + L.tok);
    int32_t* hpos = reinterpret_cast<int32_t*>(hb + L.pos);
    int64_t* hslot = reinterpret_cast<int64_t*>(hb + L.slot);
    int32_t* hkrow = reinterpret_cast<int32_t*>(hb + L.krow);
    int64_t* hkslot = reinterpret_cast<int64_t*>(hb + L.kslot);
    int4* hq = reinterpret_cast<int4*>(hb + L.qblk);
    int2* hseg = reinterpret_cast<int2*>(hb + L.seg);
    const int32_t B = arena->block_size;
    for (int32_t r = 0; r < R; ++r) {
      const int32_t n = lens[r] - st0[r];
      if (n == 0) continue;
      const Wave& w = plan->waves[wave_of[r]];
      const int32_t* tab = tables + (int64_t)r * max_blocks;
      const int64_t r0 = row_off[r], k0 = key_off[r];
      const int32_t kloc = (int32_t)(k0 - w.key_begin) + st0[r];  // key row of the first computed position
      for (int32_t i = 0; i < n; ++i) {
        const int32_t p = st0[r] + i;
        htok[r0 + i] = tokens[tok_off[r] + i];
        hpos[r0 + i] = p;
        hslot[r0 + i] = (int64_t)tab[p / B] * B + p % B;
        hkrow[r0 + i] = kloc + i;
      }
      for (int64_t t = r0 + n; t < row_off[r + 1]; ++t) {
        htok[t] = 0;
        hpos[t] = 0;
        hslot[t] = -1;
        hkrow[t] = kloc + (int32_t)(t - r0);
      }
      for (int32_t p = 0; p < lens[r]; ++p) hkslot[k0 + p] = (int64_t)tab[p / B] * B + p % B;
      for (int64_t t = k0 + lens[r]; t < key_off[r + 1]; ++t) hkslot[t] = -1;
    }
    const int QB = attn_qblock(d.dtype, d.num_q_heads / d.num_kv_heads);
    int32_t nq_total = 0, ns_total = 0;
    for (size_t wi = 0; wi < plan->waves.size(); ++wi) {
      Wave& w = plan->waves[wi];
      w.qblk_begin = nq_total;
      w.seg_begin = ns_total;
      std::vector<int4> blocks;
      for (int32_t r = 0; r < R; ++r) {
        if (wave_of[r] != (int32_t)wi) continue;
        const int32_t n = lens[r] - st0[r];
        const int32_t rs = (int32_t)(row_off[r] - w.tok_begin), ks = (int32_t)(key_off[r] - w.key_begin);
        for (int32_t qs = 0; qs < n; qs += QB)
          blocks.push_back(make_int4(rs + qs, std::min(QB, n - qs), ks, st0[r] + qs));
        if (n == 0 || st0[r] == 0) continue;
        for (int32_t p0 = 0; p0 < st0[r]; p0 += GATHER_KEYS)
          hseg[ns_total++] = make_int2(ks + p0, std::min(GATHER_KEYS, st0[r] - p0));
        // key rows past the computed ones up to the 64-aligned region end:
        // zeros (a negative count), since the last key tile reads them
        const int32_t kend = st0[r] + (int32_t)(row_off[r + 1] - row_off[r]);
        const int32_t ktot = (int32_t)(key_off[r + 1] - key_off[r]);
        if (ktot > kend) hseg[ns_total++] = make_int2(ks + kend, -(ktot - kend));
      }
      // longest causal extent first
      std::stable_sort(blocks.begin(), blocks.end(),
                       [](const int4& x, const int4& y) { return (x.w + x.y) > (y.w + y.y); });
      std::memcpy(hq + nq_total, blocks.data(), sizeof(int4) * blocks.size());
      w.num_qblk = (int32_t)blocks.size();
      w.num_seg = ns_total - w.seg_begin;
      nq_total += w.num_qblk;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(plan->ws, hb, L.meta_end, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipEventRecord(arena->staged, s);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      delete plan;
      return fail(KV_EDEVICE, "metadata upload failed: %s", hipGetErrorString(e));
    }
    arena->staged_pending = true;
  }
  {
    std::lock_guard<std::mutex> g(g_reg_mu);
    g_plans.insert(plan);
  }
  *out = plan;
  return ok();
}

}  // namespace

extern "C" {

kv_status kv_rebuild_stage(kv_arena_t arena, const int32_t* tokens, const int32_t* lens, int32_t R,
                           const int32_t* tables, int32_t max_blocks, void* workspace,
                           uint64_t ws_bytes, void* stream, kv_plan_t* out) {
  return stage_impl(arena, tokens, lens, nullptr, R, tables, max_blocks, workspace, ws_bytes, stream,
                    out);
}

kv_status kv_rebuild_stage_from(kv_arena_t arena, const int32_t* tokens, const int32_t* lens,
                                const int32_t* starts, int32_t R, const int32_t* tables,
                                int32_t max_blocks, void* workspace, uint64_t ws_bytes, void* stream,
                                kv_plan_t* out) {
  if (R > 0 && !starts) return fail(KV_EINVAL, "null starts");
  return stage_impl(arena, tokens, lens, starts, R, tables, max_blocks, workspace, ws_bytes, stream,
                    out);
}

kv_status kv_plan_release(kv_plan_t plan) {
  {
    std::lock_guard<std::mutex> g(g_reg_mu);
    if (!plan || !g_plans.count(plan)) return fail(KV_ESTATE, "unknown or released plan");
    g_plans.erase(plan);
  }
  delete plan;
  return ok();
}

kv_status kv_plan_info(kv_plan_t plan, int32_t* num_waves, int64_t* max_wave_tokens) {
  if (!live_plan(plan)) return fail(KV_ESTATE, "unknown or released plan");
  int64_t mx = 0;
  for (auto& w : plan->waves) mx = std::max<int64_t>(mx, w.rows);
  if (num_waves) *num_waves = (int32_t)plan->waves.size();
  if (max_wave_tokens) *max_wave_tokens = mx;
  return ok();
}

kv_status kv_rebuild_execute(const kv_weights* w, kv_plan_t plan, void* stream) {
  if (!live_plan(plan)) return fail(KV_ESTATE, "unknown or released plan");
  kv_arena* ar = plan->arena;
  if (!live_arena(ar)) return fail(KV_ESTATE, "the plan's arena was released");
  if (!w || !w->embed || !w->layers) return fail(KV_EINVAL, "null weights");
  const kv_model_desc& d = ar->desc;
  if (!same_desc(w->desc, d)) return fail(KV_ESTATE, "weights and arena describe different models");
  for (int l = 0; l < d.num_layers; ++l) {
    const kv_layer_weights& lw = w->layers[l];
    if (!lw.attn_norm || !lw.wq || !lw.wk || !lw.wv || !lw.wo || !lw.ffn_norm || !lw.w_gate ||
        !lw.w_up || !lw.w_down)
      return fail(KV_EINVAL, "null weight pointer in layer %d", l);
    if (d.qk_norm && (!lw.q_norm || !lw.k_norm))
      return fail(KV_EINVAL, "qk_norm model without q_norm/k_norm in layer %d", l);
    if (d.qkv_bias && (!lw.bq || !lw.bk || !lw.bv))
      return fail(KV_EINVAL, "qkv_bias model without bq/bk/bv in layer %d", l);
  }
  if (plan->waves.empty()) return ok();
  DeviceGuard dg(ar->device);
  if (dg.err != hipSuccess) return fail(KV_EDEVICE, "cannot select device %d", ar->device);
  {
    const hipError_t pre = hipGetLastError();
    if (pre != hipSuccess) return fail(KV_EDEVICE, "pending device error: %s", hipGetErrorString(pre));
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const Layout& L = plan->lay;
  char* ws = plan->ws;
  const int dt = d.dtype;
  const int64_t e = elem_bytes(dt);
  const int H = d.hidden, nq = d.num_q_heads, nkv = d.num_kv_heads, hd = d.head_dim, F = d.ffn_dim;
  const float eps = (float)d.rms_eps;
  const int64_t plane = ar->num_blocks * (int64_t)ar->block_size * nkv * hd;  // elements
  char* abase = reinterpret_cast<char*>(ar->base);
  float2* rope = reinterpret_cast<float2*>(ws + L.rope);
  float* X = reinterpret_cast<float*>(ws + L.x);
  void* A = ws + L.a;
  void* Q = ws + L.q;
  void* U = ws + L.u;
  void* VT = dt == KV_BF16 ? (void*)(ws + L.vt) : nullptr;
  void* KC = dt == KV_BF16 ? (void*)(ws + L.kc) : nullptr;
  void* HF = ws + L.hf;
  auto gemm = dt == KV_BF16 ? launch_gemm_bf16 : launch_gemm_f32;

  {
    ProfScope ps(ar, s, KV_PROF_ROPE, 0.0);
    launch_rope_table(rope, plan->max_len, hd, d.rope_theta, s);
  }
  for (const Wave& wv : plan->waves) {
    const int M = wv.rows;
    const int32_t* tok = reinterpret_cast<const int32_t*>(ws + L.tok) + wv.tok_begin;
    const int32_t* pos = reinterpret_cast<const int32_t*>(ws + L.pos) + wv.tok_begin;
    const int64_t* slot = reinterpret_cast<const int64_t*>(ws + L.slot) + wv.tok_begin;
    const int32_t* krow = plan->has_prefix ? reinterpret_cast<const int32_t*>(ws + L.krow) + wv.tok_begin : nullptr;
    const int64_t* kslot = reinterpret_cast<const int64_t*>(ws + L.kslot) + wv.key_begin;
    const int4* qblk = reinterpret_cast<const int4*>(ws + L.qblk) + wv.qblk_begin;
    const int2* segs = reinterpret_cast<const int2*>(ws + L.seg) + wv.seg_begin;
    {
      ProfScope ps(ar, s, KV_PROF_NORM, 0.0);
      launch_embed_norm(dt, w->embed, tok, w->layers[0].attn_norm, X, A, M, H, eps, s);
    }
    for (int l = 0; l < d.num_layers; ++l) {
      const kv_layer_weights& lw = w->layers[l];
      const bool last = l == d.num_layers - 1;
      if (l > 0) {
        ProfScope ps(ar, s, KV_PROF_NORM, 0.0);
        launch_rmsnorm(dt, X, lw.attn_norm, A, M, H, eps, s);
      }
      char* plane_k = abase + (int64_t)(2 * l) * plane * e;
      char* plane_v = abase + (int64_t)(2 * l + 1) * plane * e;

      GemmParams g{};
      g.A = A;
      g.lda = H;
      g.M = M;
      g.K = H;
      g.B0 = lw.wq;
      g.B1 = lw.wk;
      g.B2 = lw.wv;
      g.bmap = BMAP_QKV;
      g.s0 = nq * hd;
      g.s1 = nq * hd + nkv * hd;
      g.n_begin = last ? nq * hd : 0;
      g.n_end = (nq + 2 * nkv) * hd;
      g.epi.q_out = Q;
      g.epi.arena_k = plane_k;
      g.epi.arena_v = plane_v;
      g.epi.vt = VT;
      g.epi.kc = KC;
      g.epi.ldvt = L.Wkpad;
      g.epi.krow = krow;
      g.epi.slot = slot;
      g.epi.pos = pos;
      g.epi.rope = rope;
      g.epi.nq = nq;
      g.epi.nkv = nkv;
      g.epi.d = hd;
      g.epi.bq = d.qkv_bias ? lw.bq : nullptr;
      g.epi.bk = d.qkv_bias ? lw.bk : nullptr;
      g.epi.bv = d.qkv_bias ? lw.bv : nullptr;
      g.epi.q_norm = d.qk_norm ? lw.q_norm : nullptr;
      g.epi.k_norm = d.qk_norm ? lw.k_norm : nullptr;
      g.epi.eps = eps;
      {
        ProfScope ps(ar, s, KV_PROF_GEMM_QKV, 2.0 * wv.tokens * (double)(g.n_end - g.n_begin) * H);
        gemm(EPI_QKV, g, s);
      }
      if (last) break;
      if (wv.num_seg > 0 && dt == KV_BF16) {
        // retained prefix keys of this layer into the K copy and V^T
        ProfScope ps(ar, s, KV_PROF_ATTN, 0.0);
        launch_prefix_gather(segs, wv.num_seg, kslot, plane_k, plane_v, KC, VT, L.Wkpad, nkv, hd, s);
      }

      AttnParams ap{};
      ap.q = Q;
      ap.arena_k = plane_k;
      ap.arena_v = plane_v;
      ap.vt = VT;
      ap.kc = KC;
      ap.ldvt = L.Wkpad;
      ap.kslot = kslot;
      ap.qblk = qblk;
      ap.num_qblk = wv.num_qblk;
      ap.out = U;
      ap.nq = nq;
      ap.nkv = nkv;
      ap.d = hd;
      {
        // causal-triangle flops: QK^T and PV over the visible (query, key) pairs
        ProfScope ps(ar, s, KV_PROF_ATTN, 4.0 * nq * hd * wv.causal_pairs);
        if (dt == KV_BF16) launch_attention_bf16(ap, s); else launch_attention_f32(ap, M, s);
      }

      GemmParams go{};
      go.A = U;
      go.lda = nq * hd;
      go.M = M;
      go.K = nq * hd;
      go.B0 = lw.wo;
      go.bmap = BMAP_PLAIN;
      go.n_begin = 0;
      go.n_end = H;
      go.epi.x = X;
      go.epi.ldx = H;
      {
        ProfScope ps(ar, s, KV_PROF_GEMM_O, 2.0 * wv.tokens * (double)H * nq * hd);
        gemm(EPI_RESID, go, s);
      }
      {
        ProfScope ps(ar, s, KV_PROF_NORM, 0.0);
        launch_rmsnorm(dt, X, lw.ffn_norm, A, M, H, eps, s);
      }
      GemmParams gu{};
      gu.A = A;
      gu.lda = H;
      gu.M = M;
      gu.K = H;
      gu.B0 = lw.w_gate;
      gu.B1 = lw.w_up;
      gu.bmap = BMAP_GATEUP;
      gu.n_begin = 0;
      gu.n_end = 2 * F;
      gu.epi.hf = HF;
      gu.epi.ldh = F;
      gu.epi.ffn = F;
      {
        ProfScope ps(ar, s, KV_PROF_GEMM_GATEUP, 2.0 * wv.tokens * 2.0 * F * H);
        gemm(EPI_SWIGLU, gu, s);
      }
      GemmParams gd{};
      gd.A = HF;
      gd.lda = F;
      gd.M = M;
      gd.K = F;
      gd.B0 = lw.w_down;
      gd.bmap = BMAP_PLAIN;
      gd.n_begin = 0;
      gd.n_end = H;
      gd.epi.x = X;
      gd.epi.ldx = H;
      {
        ProfScope ps(ar, s, KV_PROF_GEMM_DOWN, 2.0 * wv.tokens * (double)H * F);
        gemm(EPI_RESID, gd, s);
      }
    }
  }
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(KV_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
  return ok();
}

kv_status kv_rebuild_from_check(const kv_model_desc* desc, int32_t block_size, int64_t num_blocks,
                                const int32_t* tokens, const int32_t* lens, const int32_t* starts,
                                int32_t num_requests, const int32_t* block_tables,
                                int32_t max_blocks_per_req) {
  if (num_requests > 0 && !starts) return fail(KV_EINVAL, "null starts");
  kv_status st = check_request(desc, block_size, num_blocks, tokens, lens, num_requests, block_tables,
                               max_blocks_per_req, nullptr, nullptr, starts);
  return st == KV_OK ? ok() : st;
}

kv_status kv_rebuild_from(const kv_weights* w, const int32_t* tokens, const int32_t* lens,
                          const int32_t* starts, int32_t R, const int32_t* tables, int32_t max_blocks,
                          kv_arena_t arena, void* workspace, uint64_t ws_bytes, void* stream) {
  if (!w) return fail(KV_EINVAL, "null weights");
  if (!live_arena(arena)) return fail(KV_ESTATE, "unknown or released arena handle");
  if (!same_desc(w->desc, arena->desc)) return fail(KV_ESTATE, "weights and arena describe different models");
  kv_plan_t plan = nullptr;
  kv_status st = kv_rebuild_stage_from(arena, tokens, lens, starts, R, tables, max_blocks, workspace,
                                       ws_bytes, stream, &plan);
  if (st != KV_OK) return st;
  st = kv_rebuild_execute(w, plan, stream);
  const std::string keep = g_err;
  kv_plan_release(plan);
  if (st != KV_OK) {
    g_err = keep;
    return st;
  }
  return ok();
}

kv_status kv_rebuild(const kv_weights* w, const int32_t* tokens, const int32_t* lens, int32_t R,
                     const int32_t* tables, int32_t max_blocks, kv_arena_t arena, void* workspace,
                     uint64_t ws_bytes, void* stream) {
  if (!w) return fail(KV_EINVAL, "null weights");
  if (!live_arena(arena)) return fail(KV_ESTATE, "unknown or released arena handle");
  if (!same_desc(w->desc, arena->desc)) return fail(KV_ESTATE, "weights and arena describe different models");
  kv_plan_t plan = nullptr;
  kv_status st = kv_rebuild_stage(arena, tokens, lens, R, tables, max_blocks, workspace, ws_bytes,
                                  stream, &plan);
  if (st != KV_OK) return st;
  st = kv_rebuild_execute(w, plan, stream);
  const std::string keep = g_err;
  kv_plan_release(plan);
  if (st != KV_OK) {
    g_err = keep;
    return st;
  }
  return ok();
}

// ---------------------------------------------------------------------------
// Resumed decode (kvr_decode.h)
// ---------------------------------------------------------------------------
uint64_t kv_decode_workspace_bytes(const kv_model_desc* desc, int32_t num_requests,
                                   int64_t max_position) {
  if (check_desc(desc) != KV_OK || num_requests <= 0 || max_position <= 0) return 0;
  return make_decode_layout(*desc, num_requests, max_position).total;
}

kv_status kv_decode_check(const kv_model_desc* desc, int32_t block_size, int64_t num_blocks,
                          const int32_t* tokens, const int32_t* positions, int32_t num_requests,
                          const int32_t* block_tables, int32_t max_blocks_per_req) {
  kv_status st = check_decode(desc, block_size, num_blocks, tokens, positions, num_requests,
                              block_tables, max_blocks_per_req, nullptr);
  return st == KV_OK ? ok() : st;
}

kv_status kv_decode_step(const kv_weights* w, const void* final_norm, const void* lm_head,
                         const int32_t* tokens, const int32_t* positions, int32_t R,
                         const int32_t* tables, int32_t max_blocks, kv_arena_t arena,
                         void* workspace, uint64_t ws_bytes, void* stream, int32_t* next_tokens,
                         float* logits) {
  if (!live_arena(arena)) return fail(KV_ESTATE, "unknown or released arena handle");
  if (!w || !w->embed || !w->layers) return fail(KV_EINVAL, "null weights");
  const kv_model_desc& d = arena->desc;
  if (!same_desc(w->desc, d)) return fail(KV_ESTATE, "weights and arena describe different models");
  int64_t max_pos = 0;
  kv_status st = check_decode(&d, arena->block_size, arena->num_blocks, tokens, positions, R, tables,
                              max_blocks, &max_pos);
  if (st != KV_OK) return st;
  if (R == 0) return ok();
  if (!final_norm || !lm_head) return fail(KV_EINVAL, "null final_norm or lm_head");
  if (!next_tokens) return fail(KV_EINVAL, "null next_tokens");
  for (int l = 0; l < d.num_layers; ++l) {
    const kv_layer_weights& lw = w->layers[l];
    if (!lw.attn_norm || !lw.wq || !lw.wk || !lw.wv || !lw.wo || !lw.ffn_norm || !lw.w_gate ||
        !lw.w_up || !lw.w_down)
      return fail(KV_EINVAL, "null weight pointer in layer %d", l);
    if (d.qk_norm && (!lw.q_norm || !lw.k_norm))
      return fail(KV_EINVAL, "qk_norm model without q_norm/k_norm in layer %d", l);
    if (d.qkv_bias && (!lw.bq || !lw.bk || !lw.bv))
      return fail(KV_EINVAL, "qkv_bias model without bq/bk/bv in layer %d", l);
  }
  if (!workspace) return fail(KV_EINVAL, "null workspace");
  const DecodeLayout L = make_decode_layout(d, R, max_pos + 1);
  if (L.total > ws_bytes)
    return fail(KV_ENOMEM, "workspace of %llu bytes < %llu needed", (unsigned long long)ws_bytes,
                (unsigned long long)L.total);
  DeviceGuard dg(arena->device);
  if (dg.err != hipSuccess) return fail(KV_EDEVICE, "cannot select device %d", arena->device);
  {
    const hipError_t pre = hipGetLastError();
    if (pre != hipSuccess) return fail(KV_EDEVICE, "pending device error: %s", hipGetErrorString(pre));
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* ws = reinterpret_cast<char*>(workspace);
  const int32_t B = arena->block_size;

  // ---- stage metadata through the arena's pinned buffer ----
  if (arena->staged_pending) {
    (void)hipEventSynchronize(arena->staged);
    arena->staged_pending = false;
  }
  if (arena->pinned_bytes < L.meta_end) {
    if (arena->pinned) (void)hipHostFree(arena->pinned);
    arena->pinned = nullptr;
    arena->pinned_bytes = 0;
    if (hipHostMalloc(&arena->pinned, L.meta_end, hipHostMallocDefault) != hipSuccess) {
      arena->pinned = nullptr;
      return fail(KV_ENOMEM, "pinned staging allocation of %zu bytes failed", (size_t)L.meta_end);
    }
    arena->pinned_bytes = L.meta_end;
  }
  char* hb = reinterpret_cast<char*>(arena->pinned);
  int32_t* htok = reinterpret_cast<int32_t*>(hb + L.tok);
  int32_t* hpos = reinterpret_cast<int32_t*>(hb + L.pos);
  int32_t* hrow = reinterpret_cast<int32_t*>(hb + L.rowidx);
  int64_t* hslot = reinterpret_cast<int64_t*>(hb + L.slot);
  int32_t* hctx = reinterpret_cast<int32_t*>(hb + L.ctx);
  int32_t* htab = reinterpret_cast<int32_t*>(hb + L.tables);
  const int32_t tab_ld = (int32_t)(max_pos / B + 1);  // staged table entries per request
  for (int32_t r = 0; r < R; ++r) {
    const int32_t p = positions[r];
    const int32_t* tab = tables + (int64_t)r * max_blocks;
    htok[r] = tokens[r];
    hpos[r] = p;
    hrow[r] = r;
    hslot[r] = (int64_t)tab[p / B] * B + p % B;
    hctx[r] = p + 1;
    for (int32_t b = 0; b < tab_ld; ++b) htab[(int64_t)r * tab_ld + b] = b <= p / B ? tab[b] : 0;
  }
  {
    const size_t meta_bytes = L.tables + (size_t)4 * R * tab_ld;
    hipError_t e = hipMemcpyAsync(ws, hb, meta_bytes, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipEventRecord(arena->staged, s);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(KV_EDEVICE, "metadata upload failed: %s", hipGetErrorString(e));
    }
    arena->staged_pending = true;
  }

  const int dt = d.dtype;
  const int64_t e = elem_bytes(dt);
  const int H = d.hidden, nq = d.num_q_heads, nkv = d.num_kv_heads, hd = d.head_dim, F = d.ffn_dim;
  const float eps = (float)d.rms_eps;
  const int64_t plane = arena->num_blocks * (int64_t)B * nkv * hd;  // elements
  char* abase = reinterpret_cast<char*>(arena->base);
  const int32_t* d_tok = reinterpret_cast<const int32_t*>(ws + L.tok);
  const int32_t* d_pos = reinterpret_cast<const int32_t*>(ws + L.pos);
  const int32_t* d_row = reinterpret_cast<const int32_t*>(ws + L.rowidx);
  const int64_t* d_slot = reinterpret_cast<const int64_t*>(ws + L.slot);
  const int32_t* d_ctx = reinterpret_cast<const int32_t*>(ws + L.ctx);
  const int32_t* d_tab = reinterpret_cast<const int32_t*>(ws + L.tables);
  float2* rope = reinterpret_cast<float2*>(ws + L.rope);
  float* X = reinterpret_cast<float*>(ws + L.x);
  void* A = ws + L.a;
  void* Q = ws + L.q;
  void* U = ws + L.u;
  void* HF = ws + L.hf;
  float* part = reinterpret_cast<float*>(ws + L.part);
  float* gpart = reinterpret_cast<float*>(ws + L.gpart);
  float2* amax = reinterpret_cast<float2*>(ws + L.amax);
  float* logit_t = reinterpret_cast<float*>(ws + L.logit);
  (void)e;
  // few rows: bf16 products split K across the chip (fp32 partials summed in
  // a fixed order); fp32 products are small enough for the plain kernel
  auto gemm = [&](int epi, const GemmParams& gp, hipStream_t st) {
    if (dt == KV_BF16)
      launch_gemm_bf16_splitk(epi, gp, gpart, L.gpart_elems, st);
    else
      launch_gemm_f32(epi, gp, st);
  };
  auto gemm_full = dt == KV_BF16 ? launch_gemm_bf16 : launch_gemm_f32;
  // a residual product and the RMSNorm of the updated rows with `gain`: one
  // kernel after the bf16 few-row product, else the product and the norm
  auto resid_norm = [&](const GemmParams& gp, const void* gain) {
    if (dt == KV_BF16 && launch_gemm_bf16_splitk_resid_norm(gp, gpart, L.gpart_elems, gain, A, eps, s))
      return;
    gemm(EPI_RESID, gp, s);
    launch_rmsnorm(dt, X, gain, A, R, H, eps, s);
  };

  // rope rows of the step's positions; the QKV epilogue indexes them by row
  launch_rope_rows(rope, d_pos, R, hd, d.rope_theta, s);
  launch_embed_norm(dt, w->embed, d_tok, w->layers[0].attn_norm, X, A, R, H, eps, s);
  for (int l = 0; l < d.num_layers; ++l) {
    const kv_layer_weights& lw = w->layers[l];
    char* plane_k = abase + (int64_t)(2 * l) * plane * elem_bytes(dt);
    char* plane_v = abase + (int64_t)(2 * l + 1) * plane * elem_bytes(dt);
    GemmParams g{};
    g.A = A;
    g.lda = H;
    g.M = R;
    g.K = H;
    g.B0 = lw.wq;
    g.B1 = lw.wk;
    g.B2 = lw.wv;
    g.bmap = BMAP_QKV;
    g.s0 = nq * hd;
    g.s1 = nq * hd + nkv * hd;
    g.n_begin = 0;
    g.n_end = (nq + 2 * nkv) * hd;
    g.epi.q_out = Q;
    g.epi.arena_k = plane_k;
    g.epi.arena_v = plane_v;
    g.epi.vt = nullptr;
    g.epi.kc = nullptr;
    g.epi.ldvt = 0;
    g.epi.slot = d_slot;
    g.epi.pos = d_row;
    g.epi.rope = rope;
    g.epi.nq = nq;
    g.epi.nkv = nkv;
    g.epi.d = hd;
    g.epi.bq = d.qkv_bias ? lw.bq : nullptr;
    g.epi.bk = d.qkv_bias ? lw.bk : nullptr;
    g.epi.bv = d.qkv_bias ? lw.bv : nullptr;
    g.epi.q_norm = d.qk_norm ? lw.q_norm : nullptr;
    g.epi.k_norm = d.qk_norm ? lw.k_norm : nullptr;
    g.epi.eps = eps;
    gemm(EPI_QKV, g, s);

    DecodeAttnParams ap{};
    ap.q = Q;
    ap.plane_k = plane_k;
    ap.plane_v = plane_v;
    ap.tables = d_tab;
    ap.max_blocks = tab_ld;
    ap.block_size = B;
    ap.ctx = d_ctx;
    ap.nq = nq;
    ap.nkv = nkv;
    ap.d = hd;
    ap.splits = decode_attn_splits(R, nkv, max_pos + 1);
    ap.part = part;
    ap.out = U;
    launch_decode_attention(dt, ap, R, s);

    GemmParams go{};
    go.A = U;
    go.lda = nq * hd;
    go.M = R;
    go.K = nq * hd;
    go.B0 = lw.wo;
    go.bmap = BMAP_PLAIN;
    go.n_begin = 0;
    go.n_end = H;
    go.epi.x = X;
    go.epi.ldx = H;
    resid_norm(go, lw.ffn_norm);
    GemmParams gu{};
    gu.A = A;
    gu.lda = H;
    gu.M = R;
    gu.K = H;
    gu.B0 = lw.w_gate;
    gu.B1 = lw.w_up;
    gu.bmap = BMAP_GATEUP;
    gu.n_begin = 0;
    gu.n_end = 2 * F;
    gu.epi.hf = HF;
    gu.epi.ldh = F;
    gu.epi.ffn = F;
    gemm(EPI_SWIGLU, gu, s);
    GemmParams gd{};
    gd.A = HF;
    gd.lda = F;
    gd.M = R;
    gd.K = F;
    gd.B0 = lw.w_down;
    gd.bmap = BMAP_PLAIN;
    gd.n_begin = 0;
    gd.n_end = H;
    gd.epi.x = X;
    gd.epi.ldx = H;
    // the next layer's attention norm, or the final norm after the last layer
    resid_norm(gd, l + 1 < d.num_layers ? w->layers[l + 1].attn_norm : final_norm);
  }
  // LM head over the final-normed rows (the last layer's residual step wrote
  // them), argmax.  bf16: the few-row product writes row-major logits (into
  // the caller's buffer when one is given); otherwise, and where the
  // vocabulary is not a multiple of its blocks, the transposed product (vocab
  // rows x padded request columns)
  if (dt == KV_BF16) {
    GemmParams gr{};
    gr.A = A;
    gr.lda = H;
    gr.M = R;
    gr.K = H;
    gr.B0 = lm_head;
    gr.bmap = BMAP_PLAIN;
    gr.n_begin = 0;
    gr.n_end = d.vocab;
    float* out = logits ? logits : logit_t;
    if (launch_gemm_bf16_rows(gr, out, d.vocab, s)) {
      launch_argmax_rows(out, d.vocab, d.vocab, R, amax, next_tokens, s);
      const hipError_t err = hipGetLastError();
      if (err != hipSuccess) return fail(KV_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
      return ok();
    }
  }
  GemmParams gl{};
  gl.A = lm_head;
  gl.lda = H;
  gl.M = d.vocab;
  gl.K = H;
  gl.B0 = A;
  gl.ldb = H;
  gl.bmap = BMAP_PLAIN;
  gl.n_begin = 0;
  gl.n_end = dt == KV_BF16 ? L.npad : R;
  gl.epi.x = logit_t;
  gl.epi.ldx = L.npad;
  gemm_full(EPI_STORE, gl, s);
  launch_argmax(logit_t, L.npad, d.vocab, R, amax, next_tokens, logits, s);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(KV_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
  return ok();
}

// ---------------------------------------------------------------------------
// Block commit digests and verification (kvr_verify.h)
// ---------------------------------------------------------------------------
}  // extern "C"

namespace {

// Workspace: the staged entry list (block, covered slots) and request offsets,
// then the per-entry match flags and a digest buffer for calls that do not
// want the digests back.
struct VerifyLayout {
  size_t entries = 0, offsets = 0, meta_end = 0, match = 0, digests = 0, total = 0;
};

VerifyLayout make_verify_layout(int32_t R, int64_t E) {
  VerifyLayout L;
  size_t off = 0;
  auto seg = [&](size_t bytes) {
    const size_t at = off;
    off = (size_t)round_up((int64_t)(off + bytes), 256);
    return at;
  };
  L.entries = seg(8 * (size_t)E);
  L.offsets = seg(4 * ((size_t)R + 1));
  L.meta_end = off;
  L.match = seg((size_t)E);
  L.digests = seg(8 * (size_t)E);
  L.total = off;
  return L;
}

// Host-side checks shared by the verification entry points; *E_out receives
// the entry count.
kv_status verify_check(kv_arena* arena, const int32_t* lens, int32_t R, const int32_t* tables,
                       int32_t max_blocks, const uint64_t* committed, uint64_t* digests,
                       int32_t* intact, int64_t* E_out) {
  if (!live_arena(arena)) return fail(KV_ESTATE, "unknown or released arena handle");
  if (R < 0) return fail(KV_EINVAL, "num_requests < 0");
  if (R > 0 && (!lens || !tables)) return fail(KV_EINVAL, "null lens or block tables");
  const kv_model_desc& d = arena->desc;
  const int64_t row = (int64_t)d.num_kv_heads * d.head_dim * elem_bytes(d.dtype);
  if (row % 16 != 0) return fail(KV_EINVAL, "slot row of %lld bytes is not a multiple of 16", (long long)row);
  const int32_t B = arena->block_size;
  int64_t E = 0;
  for (int32_t r = 0; r < R; ++r) {
    if (lens[r] < 0) return fail(KV_EINVAL, "request %d has length %d", r, lens[r]);
    const int64_t nb = ((int64_t)lens[r] + B - 1) / B;
    if (nb > max_blocks)
      return fail(KV_ECAPACITY, "request %d needs %lld blocks > %d table entries", r, (long long)nb, max_blocks);
    for (int64_t j = 0; j < nb; ++j) {
      const int32_t b = tables[(int64_t)r * max_blocks + j];
      if (b < 0 || b >= arena->num_blocks)
        return fail(KV_ERANGE, "request %d block %lld is %d, outside [0, %lld)", r, (long long)j, b,
                    (long long)arena->num_blocks);
    }
    E += nb;
  }
  if (E > 0x7fffffffLL) return fail(KV_EINVAL, "more than 2^31-1 blocks");
  if (E > 0 && !committed && !digests) return fail(KV_EINVAL, "null digest output");
  if (committed && R > 0 && !intact) return fail(KV_EINVAL, "null intact output");
  *E_out = E;
  return KV_OK;
}

DigestParams digest_params(const kv_arena* arena, const int2* entries, int64_t E,
                           const uint64_t* committed, uint64_t* digests, uint8_t* match) {
  const kv_model_desc& d = arena->desc;
  const int64_t row = (int64_t)d.num_kv_heads * d.head_dim * elem_bytes(d.dtype);
  DigestParams p;
  p.arena = reinterpret_cast<const char*>(arena->base);
  p.block_bytes = (int64_t)arena->block_size * row;
  p.plane_bytes = arena->num_blocks * p.block_bytes;
  p.row_bytes = (int32_t)row;
  p.planes = 2 * d.num_layers;
  p.entries = entries;
  p.num_entries = E;
  p.committed = committed;
  p.digests = digests;
  p.match = match;
  return p;
}

kv_status verify_impl(kv_arena* arena, const int32_t* lens, int32_t R, const int32_t* tables,
                      int32_t max_blocks, const uint64_t* committed, void* workspace,
                      uint64_t ws_bytes, void* stream, uint64_t* digests, int32_t* intact) {
  int64_t E = 0;
  const kv_status cst = verify_check(arena, lens, R, tables, max_blocks, committed, digests, intact, &E);
  if (cst != KV_OK) return cst;
  const int32_t B = arena->block_size;
  if (R == 0) return ok();
  if (!workspace) return fail(KV_EINVAL, "null workspace");
  const VerifyLayout L = make_verify_layout(R, E);
  if (L.total > ws_bytes)
    return fail(KV_ENOMEM, "workspace of %llu bytes < %llu needed", (unsigned long long)ws_bytes,
                (unsigned long long)L.total);
  DeviceGuard dg(arena->device);
  if (dg.err != hipSuccess) return fail(KV_EDEVICE, "cannot select device %d", arena->device);
  {
    const hipError_t pre = hipGetLastError();
    if (pre != hipSuccess) return fail(KV_EDEVICE, "pending device error: %s", hipGetErrorString(pre));
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* ws = reinterpret_cast<char*>(workspace);

  if (arena->staged_pending) {
    (void)hipEventSynchronize(arena->staged);
    arena->staged_pending = false;
  }
  if (arena->pinned_bytes < L.meta_end) {
    if (arena->pinned) (void)hipHostFree(arena->pinned);
    arena->pinned = nullptr;
    arena->pinned_bytes = 0;
    if (hipHostMalloc(&arena->pinned, L.meta_end, hipHostMallocDefault) != hipSuccess) {
      arena->pinned = nullptr;
      return fail(KV_ENOMEM, "pinned staging allocation of %zu bytes failed", (size_t)L.meta_end);
    }
    arena->pinned_bytes = L.meta_end;
  }
  char* hb = reinterpret_cast<char*>(arena->pinned);
  int2* hent = reinterpret_cast<int2*>(hb + L.entries);
  int32_t* hoff = reinterpret_cast<int32_t*>(hb + L.offsets);
  int64_t e = 0;
  for (int32_t r = 0; r < R; ++r) {
    hoff[r] = (int32_t)e;
    const int32_t nb = (lens[r] + B - 1) / B;
    for (int32_t j = 0; j < nb; ++j, ++e)
      hent[e] = make_int2(tables[(int64_t)r * max_blocks + j], std::min(B, lens[r] - j * B));
  }
  hoff[R] = (int32_t)e;
  {
    hipError_t err = hipMemcpyAsync(ws, hb, L.meta_end, hipMemcpyHostToDevice, s);
    if (err == hipSuccess) err = hipEventRecord(arena->staged, s);
    if (err != hipSuccess) {
      (void)hipGetLastError();
      return fail(KV_EDEVICE, "metadata upload failed: %s", hipGetErrorString(err));
    }
    arena->staged_pending = true;
  }
  const DigestParams p = digest_params(arena, reinterpret_cast<const int2*>(ws + L.entries), E, committed,
                                      digests ? digests : reinterpret_cast<uint64_t*>(ws + L.digests),
                                      reinterpret_cast<uint8_t*>(ws + L.match));
  launch_block_digest(p, s);
  if (committed)
    launch_leading_intact(reinterpret_cast<const int32_t*>(ws + L.offsets), R, p.match, intact, s);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(KV_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
  return ok();
}

}  // namespace

extern "C" {

uint64_t kv_verify_workspace_bytes(int32_t num_requests, int64_t num_entries) {
  if (num_requests < 0 || num_entries < 0) return 0;
  return make_verify_layout(num_requests, num_entries).total;
}

kv_status kv_block_digests(kv_arena_t arena, const int32_t* lens, int32_t num_requests,
                           const int32_t* block_tables, int32_t max_blocks_per_req,
                           void* workspace, uint64_t workspace_bytes, void* stream,
                           uint64_t* digests) {
  return verify_impl(arena, lens, num_requests, block_tables, max_blocks_per_req, nullptr, workspace,
                     workspace_bytes, stream, digests, nullptr);
}

kv_status kv_verify(kv_arena_t arena, const int32_t* lens, int32_t num_requests,
                    const int32_t* block_tables, int32_t max_blocks_per_req,
                    const uint64_t* committed, void* workspace, uint64_t workspace_bytes,
                    void* stream, uint64_t* digests, int32_t* intact) {
  if (!committed) return fail(KV_EINVAL, "null committed digests");
  return verify_impl(arena, lens, num_requests, block_tables, max_blocks_per_req, committed,
                     workspace, workspace_bytes, stream, digests, intact);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Verification without allocation (kvr_verify.h, kv_verify_noalloc)
// ---------------------------------------------------------------------------
// The scratch memory of kv_verify_noalloc: one copy of this array per device,
// held until the process ends.  In host code its name stands for no device
// address; kernels get the address hipGetSymbolAddress returns for the
// current device, resolved once per device and kept in g_scratch.
static __device__ __align__(256) char scratch[KV_VERIFY_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
char* g_scratch[SCRATCH_MAX_DEVICES] = {};

// Device address of `device`'s scratch array; `device` must be current.
kv_status scratch_of(int device, char** out) {
  if (device < 0 || device >= SCRATCH_MAX_DEVICES)
    return fail(KV_EDEVICE, "device %d is beyond the %d devices the scratch table covers", device,
                SCRATCH_MAX_DEVICES);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch[device]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return fail(KV_EDEVICE, "cannot resolve the scratch array on device %d: %s", device,
                  hipGetErrorString(e));
    }
    g_scratch[device] = reinterpret_cast<char*>(ptr);
  }
  *out = g_scratch[device];
  return KV_OK;
}

}  // namespace

extern "C" {

kv_status kv_verify_noalloc(kv_arena_t arena, const int32_t* lens, int32_t R,
                            const int32_t* tables, int32_t max_blocks, const uint64_t* committed,
                            void* stream, uint64_t* digests, int32_t* intact) {
  if (!committed) return fail(KV_EINVAL, "null committed digests");
  int64_t E = 0;
  const kv_status cst = verify_check(arena, lens, R, tables, max_blocks, committed, digests, intact, &E);
  if (cst != KV_OK) return cst;
  if (R == 0) return ok();
  // scratch layout: lens, tables, request offsets, entries, match flags, digests
  uint64_t off = 0;
  auto seg = [&](uint64_t bytes) {
    const uint64_t at = off;
    off = (uint64_t)round_up((int64_t)(off + bytes), 256);
    return at;
  };
  const uint64_t o_lens = seg(4ull * R);
  const uint64_t o_tab = seg(4ull * R * (uint64_t)max_blocks);
  const uint64_t o_off = seg(4ull * ((uint64_t)R + 1));
  const uint64_t o_ent = seg(8ull * (uint64_t)E);
  const uint64_t o_match = seg((uint64_t)E);
  const uint64_t o_dig = digests ? off : seg(8ull * (uint64_t)E);
  if (off > KV_VERIFY_NOALLOC_SCRATCH_BYTES)
    return fail(KV_ENOMEM, "%d requests with %lld table entries each and %lld blocks need %llu bytes of "
                "scratch, more than the %u the allocation-free verification holds",
                R, (long long)max_blocks, (long long)E, (unsigned long long)off,
                (unsigned)KV_VERIFY_NOALLOC_SCRATCH_BYTES);
  DeviceGuard dg(arena->device);
  if (dg.err != hipSuccess) return fail(KV_EDEVICE, "cannot select device %d", arena->device);
  {
    const hipError_t pre = hipGetLastError();
    if (pre != hipSuccess) return fail(KV_EDEVICE, "pending device error: %s", hipGetErrorString(pre));
  }
  char* sp = nullptr;
  const kv_status sst = scratch_of(arena->device, &sp);
  if (sst != KV_OK) return sst;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  int32_t* d_lens = reinterpret_cast<int32_t*>(sp + o_lens);
  int32_t* d_tab = reinterpret_cast<int32_t*>(sp + o_tab);
  int32_t* d_off = reinterpret_cast<int32_t*>(sp + o_off);
  int2* d_ent = reinterpret_cast<int2*>(sp + o_ent);
  uint8_t* d_match = reinterpret_cast<uint8_t*>(sp + o_match);
  hipError_t err = hipMemcpyAsync(d_lens, lens, 4ull * R, hipMemcpyHostToDevice, s);
  if (err == hipSuccess)
    err = hipMemcpyAsync(d_tab, tables, 4ull * R * (uint64_t)max_blocks, hipMemcpyHostToDevice, s);
  if (err != hipSuccess) {
    (void)hipGetLastError();
    return fail(KV_EDEVICE, "metadata upload failed: %s", hipGetErrorString(err));
  }
  launch_verify_entries(d_lens, d_tab, R, max_blocks, arena->block_size, d_off, d_ent, s);
  const DigestParams p = digest_params(arena, d_ent, E, committed,
                                      digests ? digests : reinterpret_cast<uint64_t*>(sp + o_dig),
                                      d_match);
  launch_block_digest(p, s);
  launch_leading_intact(d_off, R, d_match, intact, s);
  err = hipGetLastError();
  if (err != hipSuccess) return fail(KV_EDEVICE, "kernel launch failed: %s", hipGetErrorString(err));
  return ok();
}

// ---------------------------------------------------------------------------
// Per-kernel-class timing (kvr_profile.h)
// ---------------------------------------------------------------------------
kv_status kv_profile_enable(kv_arena_t a, int32_t enable) {
  if (!live_arena(a)) return fail(KV_ESTATE, "unknown or released arena handle");
  a->profile = enable != 0;
  return ok();
}

kv_status kv_profile_read(kv_arena_t a, double* ms, int64_t* launches, double* flops,
                          int32_t n_classes) {
  if (!live_arena(a)) return fail(KV_ESTATE, "unknown or released arena handle");
  DeviceGuard dg(a->device);
  size_t fi = 0;
  for (auto& pe : a->prof_pending) {
    float t = 0.0f;
    (void)hipEventSynchronize(pe.second.second);
    (void)hipEventElapsedTime(&t, pe.second.first, pe.second.second);
    a->prof_ms[pe.first] += t;
    a->prof_launches[pe.first] += 1;
    a->prof_flops[pe.first] += fi < a->pending_flops.size() ? a->pending_flops[fi] : 0.0;
    ++fi;
    a->prof_pool.push_back(pe.second.first);
    a->prof_pool.push_back(pe.second.second);
  }
  a->prof_pending.clear();
  a->pending_flops.clear();
  for (int32_t c = 0; c < n_classes && c < KV_PROF_CLASSES; ++c) {
    if (ms) ms[c] = a->prof_ms[c];
    if (launches) launches[c] = a->prof_launches[c];
    if (flops) flops[c] = a->prof_flops[c];
  }
  return ok();
}

kv_status kv_profile_reset(kv_arena_t a) {
  if (!live_arena(a)) return fail(KV_ESTATE, "unknown or released arena handle");
  double tmp[KV_PROF_CLASSES];
  kv_status st = kv_profile_read(a, tmp, nullptr, nullptr, KV_PROF_CLASSES);
  if (st != KV_OK) return st;
  for (int c = 0; c < KV_PROF_CLASSES; ++c) {
    a->prof_ms[c] = 0.0;
    a->prof_launches[c] = 0;
    a->prof_flops[c] = 0.0;
  }
  return ok();
}

}  // extern "C"
