// Host-only planner: status strings, thread-local errors, CU partition,
// batch metadata, attention work lists and the workspace layout.
#include "plan.h"
#include "decode_policy.h"
#include "skinny_policy.h"

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <numeric>

namespace hs {

namespace {
thread_local std::string g_error;
}

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
}

hs_status fail(hs_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return s;
}

void clear_error() { g_error.clear(); }

const char* last_error_cstr() { return g_error.c_str(); }

hs_status validate_cfg(const hs_layer_cfg* c) {
  if (!c) return fail(HS_ERR_INVALID_ARG, "layer config is null");
  if (c->hidden <= 0 || c->hidden % 256 != 0 || c->hidden > 8192)
    return fail(HS_ERR_UNSUPPORTED, "hidden %d must be a positive multiple of 256, at most 8192", c->hidden);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(HS_ERR_UNSUPPORTED, "head_dim %d must be 64 or 128", c->head_dim);
  if (c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->n_q_heads % c->n_kv_heads != 0)
    return fail(HS_ERR_INVALID_ARG, "n_q_heads %d must be a positive multiple of n_kv_heads %d",
                c->n_q_heads, c->n_kv_heads);
  if (c->n_q_heads / c->n_kv_heads > 8)
    return fail(HS_ERR_UNSUPPORTED, "query heads per key/value head %d exceeds 8",
                c->n_q_heads / c->n_kv_heads);
  if (((c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim) % 256 != 0)
    return fail(HS_ERR_UNSUPPORTED, "(Hq + 2 Hkv) * head_dim must be a multiple of 256");
  // Hq * head_dim is the K of the output projection; the prefill GEMM walks K
  // in groups of four 32-wide stages.
  if ((c->n_q_heads * c->head_dim) % 128 != 0)
    return fail(HS_ERR_UNSUPPORTED, "Hq * head_dim must be a multiple of 128");
  if (c->ffn <= 0 || c->ffn % 128 != 0)
    return fail(HS_ERR_UNSUPPORTED, "ffn %d must be a positive multiple of 128", c->ffn);
  if (!(c->rms_eps > 0.0f) || !(c->rope_base > 1.0f))
    return fail(HS_ERR_INVALID_ARG, "rms_eps must be > 0 and rope_base > 1");
  const int32_t* sec = c->mrope_sections;
  if (sec[0] || sec[1] || sec[2]) {
    if (sec[0] < 0 || sec[1] < 0 || sec[2] < 0 || sec[0] % 4 || sec[1] % 4 || sec[2] % 4 ||
        sec[0] + sec[1] + sec[2] != c->head_dim / 2)
      return fail(HS_ERR_INVALID_ARG, "mrope_sections (%d, %d, %d) must be multiples of 4 summing to head_dim / 2",
                  sec[0], sec[1], sec[2]);
  }
  return HS_OK;
}

hs_status validate_batch(const int32_t* off, const int32_t* ctx, int32_t B, int32_t* n_tokens,
                         int32_t* max_pos) {
  if (!off) return fail(HS_ERR_INVALID_ARG, "seq_offsets is null");
  if (B < 1) return fail(HS_ERR_INVALID_ARG, "n_seqs %d must be >= 1", B);
  if (off[0] != 0) return fail(HS_ERR_INVALID_ARG, "seq_offsets[0] = %d, expected 0", off[0]);
  int64_t mp = 0;
  for (int32_t b = 0; b < B; ++b) {
    if (off[b + 1] < off[b])
      return fail(HS_ERR_INVALID_ARG, "seq_offsets decrease at %d (%d -> %d)", b, off[b], off[b + 1]);
    const int64_t c = ctx ? ctx[b] : 0;
    if (c < 0) return fail(HS_ERR_INVALID_ARG, "ctx_lens[%d] = %lld is negative", b, (long long)c);
    const int64_t end = c + (off[b + 1] - off[b]);
    if (end > (int64_t(1) << 30)) return fail(HS_ERR_UNSUPPORTED, "position too large in sequence %d", b);
    mp = std::max(mp, end);
  }
  if (off[B] <= 0) return fail(HS_ERR_INVALID_ARG, "batch has no rows");
  *n_tokens = off[B];
  *max_pos = int32_t(mp);
  return HS_OK;
}

hs_status check_32bit_extents(const hs_layer_cfg& c, int32_t T, int32_t max_ctx) {
  const int64_t limit = int64_t(1) << 32;  // exclusive: the resources' byte count is a uint32
  const int64_t d = c.hidden, f = c.ffn, qd = int64_t(c.n_q_heads) * c.head_dim;
  const int64_t qkv = int64_t(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  const struct {
    const char* what;
    int64_t bytes;
  } ext[] = {
      {"w_qkv", qkv * d * 2},          {"w_o", d * qd * 2},
      {"w_gate_up", 2 * f * d * 2},    {"w_down", d * f * 2},
      {"the hidden-wide activations", int64_t(T) * d * 2},
      {"the attention output", int64_t(T) * qd * 2},
      {"the SwiGLU output", int64_t(T) * f * 2},
  };
  for (const auto& e : ext)
    if (e.bytes >= limit)
      return fail(HS_ERR_UNSUPPORTED, "%s would take %lld bytes; the kernels address at most 2^32 - 1", e.what,
                  (long long)e.bytes);
  if (int64_t(max_ctx) * c.head_dim * 2 > 0x7ffffff0)
    return fail(HS_ERR_UNSUPPORTED, "a cache page of %d positions exceeds the 2 GiB a single-row attention unit addresses",
                max_ctx);
  return HS_OK;
}

int64_t max_att_items(int32_t T, int32_t B) { return int64_t(T) / kAttnBlockQ + B + 1; }

// Split-K scratch of the skinny GEMM over the four projections of a layer:
// the largest partial-sum buffer and the most weight strips of any of them.
struct SkinnyNeeds {
  size_t part_bytes = 0;
  int32_t counters = 0;
};

static SkinnyNeeds skinny_needs(const hs_layer_cfg& c, int32_t T) {
  SkinnyNeeds n;
  if (T > kSkinnyMaxRows) return n;
  const int mt = skinny_m_tiles(T);
  struct G {
    int strips, ns, k;
    bool used;
  };
  const G gs[4] = {
      {skinny_strips_qkv(c.n_q_heads, c.n_kv_heads, c.head_dim), 1, c.hidden, true},
      {skinny_strips_resid(c.hidden), 1, c.n_q_heads * c.head_dim, true},
      {skinny_strips_swiglu(c.ffn), 2, c.hidden, true},
      {skinny_strips_resid(c.hidden), 1, c.ffn, true},
  };
  for (const G& g : gs) {
    if (!g.used) continue;
    const SkinnySplit sp = skinny_split(g.strips, g.k / kSkinnyBK);
    n.counters = std::max(n.counters, int32_t(g.strips));
    if (sp.splits > 1)
      n.part_bytes = std::max(n.part_bytes, size_t(g.strips) * sp.splits * skinny_partial_bytes(g.ns, mt));
  }
  return n;
}

int32_t dec_unit_keys(int dh, int32_t page_keys) {
  const int32_t split = dec_split_keys(dh);
  return page_keys > 0 ? std::gcd(split, page_keys) : split;
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Upper bound on decode work items: every single-row sequence split by the
// longest possible key range.
static int64_t max_dec_items(int32_t T, int32_t B, int32_t max_pos, int32_t unit) {
  return int64_t(std::min(T, B)) * ceil_div(max_pos, unit);
}

// Upper bound on listed pages: one per sequence without a table, else every
// page up to max_pos for every sequence.
static int64_t max_pages(int32_t B, int32_t max_pos, int32_t page_keys) {
  return page_keys > 0 ? int64_t(B) * ceil_div(max_pos, page_keys) : int64_t(B);
}

static size_t meta_bytes(int32_t T, int32_t B, int64_t pages, int64_t att, int32_t counters, int64_t dec_items,
                         int64_t dec_count) {
  size_t s = 0;
  s += align_up(size_t(T) * 4, 16);       // pos
  s += align_up(size_t(T) * 12, 16);      // pos3
  s += align_up(size_t(T) * 4, 16);       // row_seq
  s += align_up(size_t(T) * 8, 16) * 2;   // k_off, v_off
  s += align_up(size_t(B) * 4, 16) * 4;   // seq_start, seq_len, seq_ctx, seq_page0
  s += align_up(size_t(pages) * 8, 16);   // page_base
  s += align_up(size_t(att) * 8, 16);     // att items
  s += align_up(size_t(B) * 16, 16);      // single-row (decode) rows
  s += align_up(size_t(counters) * 4, 16); // split-K counters
  s += align_up(size_t(dec_items) * 32, 16); // decode work items
  s += align_up(size_t(dec_count) * 4, 16);  // decode arrival counters
  s += 16;                                   // decode work item count
  return align_up(s, kAlign);
}

WsLayout ws_layout(const hs_layer_cfg& c, int32_t T, int32_t B, int32_t max_pos, int32_t page_keys, bool packs) {
  WsLayout w{};
  const size_t d = c.hidden, hq = c.n_q_heads, hkv = c.n_kv_heads, dh = c.head_dim, f = c.ffn;
  size_t p = 0;
  auto take = [&](size_t bytes) {
    const size_t at = p;
    p = align_up(p + bytes, kAlign);
    return at;
  };
  const SkinnyNeeds sk = skinny_needs(c, T);
  const int64_t dec_items = max_dec_items(T, B, max_pos, dec_unit_keys(c.head_dim, page_keys));
  w.meta_bytes = meta_bytes(T, B, max_pages(B, max_pos, page_keys), max_att_items(T, B), sk.counters, dec_items,
                            dec_items * c.n_kv_heads);
  w.meta = take(w.meta_bytes);
  // GEMM inputs of decode-sized batches are k-group-major over padded rows.
  const size_t act_rows = T <= kSkinnyMaxRows ? size_t(skinny_k8_rows(T)) : size_t(T);
  w.n = take(act_rows * d * 2);
  w.q = take(size_t(T) * hq * dh * 2);
  // Packed keys/values: sequence b starts at the 64-aligned position
  // sum_{b' < b} round_up(len_b', 64); 64 more positions cover the last
  // tile's overhang.
  w.packed_ctx = packs ? int64_t(align_up(size_t(T) + 64 * size_t(B), 64)) + 64 : 0;
  w.kpack = take(size_t(hkv) * size_t(w.packed_ctx) * dh * 2);
  w.vpack = take(size_t(hkv) * size_t(w.packed_ctx) * dh * 2);
  w.o = take(act_rows * hq * dh * 2);
  w.h = take(size_t(T) * d * 4);
  w.a = take(act_rows * f * 2);
  w.xtmp = take(size_t(T) * d * 4);
  w.sumsq = take(size_t(T) * (d / 32) * 4);
  w.rope = take(size_t(max_pos) * (dh / 2) * 8);
  w.part_bytes = sk.part_bytes;
  w.part = take(sk.part_bytes);
  w.dec_part_bytes = size_t(dec_items) * c.n_kv_heads *
                     dec_part_floats(c.n_q_heads / c.n_kv_heads, c.head_dim) * 4;
  w.dec_part = take(w.dec_part_bytes);
  w.total = p;
  return w;
}

hs_status check_block_table(const int32_t* table, int32_t pps, int32_t n_slots, int32_t page_keys,
                            const int32_t* off, const int32_t* ctx, int32_t B) {
  if (!table) return fail(HS_ERR_INVALID_ARG, "block table is null");
  if (pps < 1) return fail(HS_ERR_INVALID_ARG, "pages_per_seq %d must be >= 1", pps);
  if (n_slots < 1) return fail(HS_ERR_INVALID_ARG, "the cache has %d slots", n_slots);
  if (page_keys < 64 || page_keys % 64 != 0)
    return fail(HS_ERR_INVALID_ARG, "page size %d must be a positive multiple of 64", page_keys);
  // writer[s]: the sequence that writes slot s in this call (-1: none);
  // reader[s]: a sequence that reaches slot s (-1: none yet), -2: several.
  std::vector<int32_t> writer(size_t(n_slots), -1), reader(size_t(n_slots), -1);
  std::vector<int32_t> seen(size_t(n_slots), -1);
  for (int32_t b = 0; b < B; ++b) {
    const int64_t cx = ctx ? ctx[b] : 0, end = cx + (off[b + 1] - off[b]);
    const int64_t n = ceil_div(end, page_keys);
    if (n > pps)
      return fail(HS_ERR_INVALID_ARG, "sequence %d reaches position %lld, beyond its %d pages of %d", b,
                  (long long)(end - 1), pps, page_keys);
    for (int64_t j = 0; j < n; ++j) {
      const int32_t s = table[int64_t(b) * pps + j];
      if (s < 0 || s >= n_slots)
        return fail(HS_ERR_INVALID_ARG, "block_table[%d][%lld] = %d outside [0, %d)", b, (long long)j, s, n_slots);
      if (seen[s] == b)
        return fail(HS_ERR_INVALID_ARG, "sequence %d lists slot %d twice", b, s);
      seen[s] = b;
      reader[s] = (reader[s] == -1 || reader[s] == b) ? b : -2;
      if (j >= cx / page_keys && end > cx) writer[s] = b;  // page j receives rows cx .. end - 1
    }
  }
  for (int32_t s = 0; s < n_slots; ++s)
    if (writer[s] >= 0 && reader[s] != writer[s])
      return fail(HS_ERR_INVALID_ARG, "slot %d receives rows of sequence %d but other sequences reach it too", s,
                  writer[s]);
  return HS_OK;
}

hs_status build_plan(const hs_layer_cfg& c, const int32_t* off, const int32_t* ctx, int32_t B,
                     const KvPlacement& kv, Plan* out, const int32_t* positions3, const PlanCapacity* cap,
                     bool bidirectional) {
  Plan& P = *out;
  hs_status st = validate_batch(off, ctx, B, &P.T, &P.max_pos);
  if (st != HS_OK) return st;
  P.B = B;
  const int64_t hkv = c.n_kv_heads, dh = c.head_dim;
  const int64_t T = P.T;

  // Attention work: multi-row sequences in 128-row query blocks, longest
  // key range first; single-row sequences take the decode path.
  struct Item { int32_t b, q0, keys; };
  std::vector<Item> att;
  std::vector<int32_t> dec_seq;
  for (int32_t b = 0; b < B; ++b) {
    const int32_t len = off[b + 1] - off[b];
    const int32_t cx = ctx ? ctx[b] : 0;
    if (len == 1) {
      dec_seq.push_back(b);
    } else {
      for (int32_t q0 = 0; q0 < len; q0 += kAttnBlockQ)
        att.push_back({b, q0, cx + (bidirectional ? len : std::min(q0 + kAttnBlockQ, len))});
    }
  }
  std::stable_sort(att.begin(), att.end(), [](const Item& x, const Item& y) { return x.keys > y.keys; });
  P.n_att_items = int32_t(att.size());
  // Longest key range first among single-row sequences as well.
  std::stable_sort(dec_seq.begin(), dec_seq.end(),
                   [&](int32_t x, int32_t y) { return (ctx ? ctx[x] : 0) > (ctx ? ctx[y] : 0); });
  P.n_dec_rows = int32_t(dec_seq.size());

  // Image layout (must match meta_bytes' order and bounds).
  size_t p = 0;
  auto take = [&](size_t bytes) {
    const size_t at = p;
    p += align_up(bytes, 16);
    return at;
  };
  P.pos = take(size_t(T) * 4);
  P.pos3 = positions3 ? take(size_t(T) * 12) : 0;
  P.row_seq = take(size_t(T) * 4);
  P.k_off = take(size_t(T) * 8);
  P.v_off = take(size_t(T) * 8);
  P.seq_start = take(size_t(B) * 4);
  P.seq_len = take(size_t(B) * 4);
  P.seq_ctx = take(size_t(B) * 4);
  if (cap && P.max_pos > cap->max_pos)
    return fail(HS_ERR_INVALID_ARG, "position %d beyond the %d positions the fixed layout holds", P.max_pos - 1,
                cap->max_pos);
  P.att_items = take(size_t(cap ? max_att_items(int32_t(T), B) : P.n_att_items) * 8);
  P.dec_rows = take(size_t(cap ? B : P.n_dec_rows) * 16);
  P.n_counters = skinny_needs(c, int32_t(T)).counters;
  P.counters = take(size_t(P.n_counters) * 4);
  // Pages: a slot, or the packed buffer, is one page per sequence; with a
  // block table every page a sequence reaches is listed.
  const bool paged = kv.cache && kv.table;
  const int64_t slot_ctx = kv.cache ? kv.max_ctx : kv.packed_ctx;
  // The attention kernels address one page of one head through a 2 GiB
  // buffer window (a cache page is bounded the same way by the caller).
  if (slot_ctx * dh * 2 > 0x7ffffff0)
    return fail(HS_ERR_UNSUPPORTED, "a key page of %lld positions exceeds the 2 GiB the attention kernels address",
                (long long)slot_ctx);
  P.page_keys = int32_t(slot_ctx);
  P.unit_keys = dec_unit_keys(int(dh), paged ? kv.max_ctx : 0);
  P.n_pages = 0;
  for (int32_t b = 0; b < B; ++b) {
    const int64_t end = (ctx ? ctx[b] : 0) + (off[b + 1] - off[b]);
    P.n_pages += paged ? int32_t(ceil_div(end, slot_ctx)) : 1;
  }
  P.seq_page0 = take(size_t(B) * 4);
  P.page_base = take(size_t(cap ? max_pages(B, cap->max_pos, cap->page_keys) : P.n_pages) * 8);
  std::vector<int32_t> dec_nsplit(dec_seq.size());
  P.n_dec_items = 0;
  for (size_t r = 0; r < dec_seq.size(); ++r) {
    dec_nsplit[r] = int32_t(ceil_div((ctx ? ctx[dec_seq[r]] : 0) + 1, P.unit_keys));
    P.n_dec_items += dec_nsplit[r];
  }
  P.cap_dec_items = cap ? max_dec_items(int32_t(T), B, cap->max_pos, P.unit_keys) : P.n_dec_items;
  if (P.n_dec_items > P.cap_dec_items) return fail(HS_ERR_INTERNAL, "decode work exceeds the fixed layout");
  P.dec_items = take(size_t(P.cap_dec_items) * 32);
  P.dec_count = take(size_t(P.cap_dec_items) * hkv * 4);
  P.dec_n = take(4);
  P.image.assign(align_up(p, kAlign), 0);

  auto i32 = [&](size_t at) { return reinterpret_cast<int32_t*>(P.image.data() + at); };
  if (positions3) memcpy(P.image.data() + P.pos3, positions3, size_t(T) * 12);
  auto i64 = [&](size_t at) { return reinterpret_cast<int64_t*>(P.image.data() + at); };

  // A page (a cache slot) holds hkv heads of slot_ctx positions.  Without a
  // table sequence b has one page: slot b, or, packed (no cache), the
  // positions from the 64-aligned base_b of one buffer of packed_ctx
  // positions, so its key tiles line up with the value tiles.  Position p of
  // a sequence lies in its page p / slot_ctx at i = p % slot_ctx: key element
  // base + i * dh of head 0, value element base + (i / 32) * 32 dh + i % 32.
  P.kv_head_stride = slot_ctx * dh;
  const int64_t slot = hkv * slot_ctx * dh;  // elements per page (K and V alike)
  constexpr int64_t VT = kv_tile_keys;
  int64_t packed_base = 0;
  int32_t page = 0;
  for (int32_t b = 0; b < B; ++b) {
    const int32_t cx = ctx ? ctx[b] : 0;
    const int32_t len = off[b + 1] - off[b];
    i32(P.seq_start)[b] = off[b];
    i32(P.seq_len)[b] = len;
    i32(P.seq_ctx)[b] = cx;
    i32(P.seq_page0)[b] = page;
    int64_t* pages = i64(P.page_base) + page;
    if (paged) {
      const int32_t n = int32_t(ceil_div(int64_t(cx) + len, slot_ctx));
      for (int32_t j = 0; j < n; ++j) pages[j] = int64_t(kv.table[int64_t(b) * kv.pages_per_seq + j]) * slot;
      page += n;
    } else {
      pages[0] = kv.cache ? int64_t(b) * slot : packed_base * dh;
      page += 1;
    }
    for (int32_t t = off[b]; t < off[b + 1]; ++t) {
      i32(P.row_seq)[t] = b;
      const int64_t pos = cx + (t - off[b]);
      const int64_t base = pages[pos / slot_ctx], i = pos % slot_ctx;
      i32(P.pos)[t] = int32_t(pos);
      i64(P.k_off)[t] = base + i * dh;
      i64(P.v_off)[t] = base + (i / VT) * VT * dh + i % VT;
    }
    if (!kv.cache) packed_base += int64_t(align_up(size_t(len), 64));
  }
  if (!kv.cache && packed_base + 64 > kv.packed_ctx)
    return fail(HS_ERR_INTERNAL, "packed keys need %lld positions, %lld planned", (long long)(packed_base + 64),
                (long long)kv.packed_ctx);
  for (int32_t i = 0; i < P.n_att_items; ++i) {
    i32(P.att_items)[2 * i] = att[i].b;
    i32(P.att_items)[2 * i + 1] = att[i].q0;
  }
  i32(P.dec_n)[0] = P.n_dec_items;
  int32_t item = 0;
  for (int32_t r = 0; r < P.n_dec_rows; ++r) {
    const int32_t b = dec_seq[r];
    int32_t* row = i32(P.dec_rows) + 4 * r;
    row[0] = off[b];
    row[1] = b;
    row[2] = 0;
    row[3] = 0;
    for (int32_t sp = 0; sp < dec_nsplit[r]; ++sp, ++item) {
      // Record layout: int32 t, n_keys, split, n_split; int64 K base, V base:
      // the page holding the split's keys (a unit never straddles pages).
      int32_t* it = i32(P.dec_items + size_t(item) * 32);
      it[0] = off[b];
      it[1] = (ctx ? ctx[b] : 0) + 1;
      it[2] = sp;
      it[3] = dec_nsplit[r];
      const int64_t base = i64(P.page_base)[i32(P.seq_page0)[b] + int64_t(sp) * P.unit_keys / slot_ctx];
      i64(P.dec_items + size_t(item) * 32 + 16)[0] = base;
      i64(P.dec_items + size_t(item) * 32 + 16)[1] = base;
    }
  }
  return HS_OK;
}

}  // namespace hs

// ---------------------------------------------------------------------------
// Host-only C entry points.

extern "C" {

const char* hs_status_string(hs_status s) {
  switch (s) {
    case HS_OK: return "HS_OK";
    case HS_ERR_INVALID_ARG: return "HS_ERR_INVALID_ARG";
    case HS_ERR_UNSUPPORTED: return "HS_ERR_UNSUPPORTED";
    case HS_ERR_BUDGET: return "HS_ERR_BUDGET";
    case HS_ERR_WORKSPACE: return "HS_ERR_WORKSPACE";
    case HS_ERR_HIP: return "HS_ERR_HIP";
    case HS_ERR_INTERNAL: return "HS_ERR_INTERNAL";
  }
  return "HS_ERR_UNKNOWN";
}

const char* hs_last_error(void) { return hs::last_error_cstr(); }

hs_status hs_default_topology(int32_t n_cus, int32_t n_xcc, hs_topology* out) {
  if (!out) return hs::fail(HS_ERR_INVALID_ARG, "topology output is null");
  if (n_cus < 1 || n_cus > 256 || n_xcc < 1 || n_xcc > hs::kMaxXcc || n_cus % n_xcc != 0)
    return hs::fail(HS_ERR_INVALID_ARG, "bad topology size %d / %d", n_cus, n_xcc);
  memset(out, 0, sizeof(*out));
  out->n_cus = n_cus;
  out->n_xcc = n_xcc;
  for (int i = 0; i < n_cus; ++i) {
    const int slot = i / n_xcc;
    out->xcc[i] = uint8_t(i % n_xcc);
    out->se[i] = uint8_t(slot % 4);
    out->cu[i] = uint8_t(slot / 4);
  }
  return HS_OK;
}

hs_status hs_cu_partition(const hs_topology* t, int32_t c, uint32_t shared[8], uint32_t down[8]) {
  if (!t || !shared || !down) return hs::fail(HS_ERR_INVALID_ARG, "null argument to hs_cu_partition");
  if (t->n_cus < 1 || t->n_cus > 256 || t->n_xcc < 1 || t->n_xcc > hs::kMaxXcc)
    return hs::fail(HS_ERR_INVALID_ARG, "bad topology (%d CUs, %d XCDs)", t->n_cus, t->n_xcc);
  if (c < 1 || c > t->n_cus) return hs::fail(HS_ERR_BUDGET, "budget %d outside [1, %d]", c, t->n_cus);
  uint32_t sh[8] = {0}, dn[8] = {0};
  bool taken[256] = {false};
  for (int x = 0; x < t->n_xcc; ++x) {
    const int want = c / t->n_xcc + (x < c % t->n_xcc ? 1 : 0);
    std::vector<int> bits;
    for (int i = 0; i < t->n_cus; ++i)
      if (t->xcc[i] == x) bits.push_back(i);
    std::sort(bits.begin(), bits.end(), [&](int a, int b) {
      if (t->cu[a] != t->cu[b]) return t->cu[a] < t->cu[b];
      if (t->se[a] != t->se[b]) return t->se[a] < t->se[b];
      return a < b;
    });
    if (int(bits.size()) < want)
      return hs::fail(HS_ERR_INVALID_ARG, "XCD %d has %d CUs, %d requested", x, int(bits.size()), want);
    for (int k = 0; k < want; ++k) taken[bits[k]] = true;
  }
  for (int i = 0; i < t->n_cus; ++i) {
    if (taken[i])
      sh[i / 32] |= 1u << (i % 32);
    else
      dn[i / 32] |= 1u << (i % 32);
  }
  memcpy(shared, sh, sizeof(sh));
  memcpy(down, dn, sizeof(dn));
  return HS_OK;
}

hs_status hs_plan_metadata(const int32_t* off, const int32_t* ctx, int32_t n_seqs, int32_t* pos_out,
                           int32_t* seq_id_out) {
  if (!pos_out || !seq_id_out) return hs::fail(HS_ERR_INVALID_ARG, "null output array");
  int32_t T = 0, mp = 0;
  hs_status st = hs::validate_batch(off, ctx, n_seqs, &T, &mp);
  if (st != HS_OK) return st;
  for (int32_t b = 0; b < n_seqs; ++b)
    for (int32_t t = off[b]; t < off[b + 1]; ++t) {
      pos_out[t] = (ctx ? ctx[b] : 0) + (t - off[b]);
      seq_id_out[t] = b;
    }
  return HS_OK;
}

hs_status hs_workspace_size(const hs_layer_cfg* cfg, int32_t max_tokens, int32_t max_seqs, int32_t max_pos,
                            size_t* bytes) {
  hs_status st = hs::validate_cfg(cfg);
  if (st != HS_OK) return st;
  if (!bytes) return hs::fail(HS_ERR_INVALID_ARG, "bytes output is null");
  if (max_tokens < 1 || max_seqs < 1 || max_pos < 1)
    return hs::fail(HS_ERR_INVALID_ARG, "sizes must be >= 1");
  *bytes = hs::ws_layout(*cfg, max_tokens, max_seqs, max_pos).total;
  return HS_OK;
}

hs_status hs_workspace_size_paged(const hs_layer_cfg* cfg, int32_t max_tokens, int32_t max_seqs, int32_t max_pos,
                                  int32_t page_positions, size_t* bytes) {
  hs_status st = hs::validate_cfg(cfg);
  if (st != HS_OK) return st;
  if (!bytes) return hs::fail(HS_ERR_INVALID_ARG, "bytes output is null");
  if (max_tokens < 1 || max_seqs < 1 || max_pos < 1)
    return hs::fail(HS_ERR_INVALID_ARG, "sizes must be >= 1");
  if (page_positions < 0 || page_positions % 64 != 0)
    return hs::fail(HS_ERR_INVALID_ARG, "page size %d must be 0 or a positive multiple of 64", page_positions);
  *bytes = hs::ws_layout(*cfg, max_tokens, max_seqs, max_pos, page_positions).total;
  return HS_OK;
}

}  // extern "C"
