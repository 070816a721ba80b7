// Host side of the Huff-LLM bf16 codec: codebooks, HLF1 encoder, validation.
//
// Huff-LLM (arXiv 2502.00922): weights are split into bit fields and each
// coded field gets its own Huffman code, once, offline, on the CPU (Sec. 3.1);
// for bf16 the split is 1-4-4-7 with the sign and mantissa kept raw
// (Sec. 5.1). The container layout and the tie rules are specified in
// include/hufflm.h.
#include "hufflm.h"
#include "hl_internal.h"

#include <sched.h>

#include <algorithm>
#include <array>
#include <cstring>
#include <functional>
#include <queue>
#include <thread>
#include <tuple>
#include <vector>

namespace hl {

// ---------------------------------------------------------------- code lengths

// Huffman lengths with the heap order (weight, kind, id); see the header.
// f and len have n entries (16 for the exponent nibbles, 256 for the whole
// exponent byte).
static void huffman_lengths(const uint64_t* f, int n, uint8_t* len) {
  using Key = std::tuple<uint64_t, int, int>;  // weight, kind (0 leaf / 1 node), id
  std::priority_queue<Key, std::vector<Key>, std::greater<Key>> heap;
  for (int s = 0; s < n; ++s) {
    len[s] = 0;
    if (f[s]) heap.emplace(f[s], 0, s);
  }
  if (heap.size() <= 1) return;
  // children of internal node id: (kind, id) pairs
  std::vector<std::array<int, 4>> kids;
  while (heap.size() > 1) {
    Key a = heap.top(); heap.pop();
    Key b = heap.top(); heap.pop();
    int id = (int)kids.size();
    kids.push_back({std::get<1>(a), std::get<2>(a), std::get<1>(b), std::get<2>(b)});
    heap.emplace(std::get<0>(a) + std::get<0>(b), 1, id);
  }
  // depth-first walk from the root
  std::vector<std::array<int, 3>> st;  // kind, id, depth
  st.push_back({std::get<1>(heap.top()), std::get<2>(heap.top()), 0});
  while (!st.empty()) {
    auto [kind, id, d] = st.back();
    st.pop_back();
    if (kind == 0) {
      len[id] = (uint8_t)d;
    } else {
      st.push_back({kids[id][0], kids[id][1], d + 1});
      st.push_back({kids[id][2], kids[id][3], d + 1});
    }
  }
}

// Package-merge lengths limited to lmax; see the header for the item order.
// Requires at most 2^lmax present symbols.
static void package_merge(const uint64_t* f, int n, int lmax, uint8_t* len) {
  struct Item { uint64_t w; int kind; std::vector<uint8_t> cnt; };
  std::vector<std::pair<uint64_t, int>> present;
  for (int s = 0; s < n; ++s) {
    len[s] = 0;
    if (f[s]) present.emplace_back(f[s], s);
  }
  std::sort(present.begin(), present.end());
  const size_t np = present.size();
  if (np <= 1) return;
  std::vector<Item> leaves;
  for (auto& p : present) {
    Item it{p.first, 0, std::vector<uint8_t>(n, 0)};
    it.cnt[p.second] = 1;
    leaves.push_back(std::move(it));
  }
  std::vector<Item> cur = leaves;
  for (int round = 0; round < lmax - 1; ++round) {
    std::vector<Item> next = leaves;
    for (size_t i = 0; i + 1 < cur.size(); i += 2) {
      Item pk{cur[i].w + cur[i + 1].w, 1, std::vector<uint8_t>(n)};
      for (int s = 0; s < n; ++s) pk.cnt[s] = (uint8_t)(cur[i].cnt[s] + cur[i + 1].cnt[s]);
      next.push_back(std::move(pk));
    }
    std::stable_sort(next.begin(), next.end(), [](const Item& a, const Item& b) {
      return a.w != b.w ? a.w < b.w : a.kind < b.kind;
    });
    cur.swap(next);
  }
  for (size_t i = 0; i < 2 * (np - 1) && i < cur.size(); ++i)
    for (int s = 0; s < n; ++s) len[s] = (uint8_t)(len[s] + cur[i].cnt[s]);
}

// Huffman lengths, replaced by package-merge lengths when longer than lmax.
static void limited_lengths(const uint64_t* f, int n, int lmax, uint8_t* len) {
  huffman_lengths(f, n, len);
  int mx = 0;
  for (int s = 0; s < n; ++s) mx = std::max(mx, (int)len[s]);
  if (mx > lmax) package_merge(f, n, lmax, len);
}

static void field_presence(const uint64_t f[16], hl_field_code* fc) {
  int nsym = 0, single = 0;
  for (int s = 0; s < 16; ++s)
    if (f[s]) { ++nsym; single = s; }
  fc->nsym = (uint8_t)nsym;
  fc->single = (uint8_t)(nsym == 1 ? single : 0);
}

// Smallest length limit a prefix code of the present symbols can meet: 0 for
// one symbol, else ceil(log2(count)).
static int min_limit(const uint64_t f[16]) {
  int n = 0;
  for (int s = 0; s < 16; ++s) n += f[s] ? 1 : 0;
  int b = 0;
  while (n > 1 && (1 << b) < n) ++b;
  return b;
}

static uint64_t code_cost(const uint64_t f[16], const uint8_t* len) {
  uint64_t c = 0;
  for (int s = 0; s < 16; ++s) c += f[s] * len[s];
  return c;
}

// The two exponent codes: each at most lmax bits and, with pair_max > 0, the
// longest eh code plus the longest el code at most pair_max bits. Every code
// pair meeting the joint limit has some longest eh code a, so it costs at
// least the optimal codes limited to a and pair_max - a: the result is the
// cheapest of those splits, a = 0 .. lmax, the smallest a on equal cost.
// False when pair_max is too small for the alphabets.
static bool pair_limited_lengths(const uint64_t feh[16], const uint64_t fel[16], int lmax, int pair_max,
                                 uint8_t leh[16], uint8_t lel[16]) {
  if (pair_max <= 0) {
    limited_lengths(feh, 16, lmax, leh);
    limited_lengths(fel, 16, lmax, lel);
    return true;
  }
  bool found = false;
  uint64_t best = 0;
  const int mh = min_limit(feh), ml = min_limit(fel);
  for (int a = 0; a <= lmax; ++a) {
    const int b = std::min(lmax, pair_max - a);
    if (b < ml) break;
    if (a < mh) continue;
    uint8_t ta[16] = {0}, tb[16] = {0};
    if (a) limited_lengths(feh, 16, a, ta);
    if (b) limited_lengths(fel, 16, b, tb);
    const uint64_t c = code_cost(feh, ta) + code_cost(fel, tb);
    if (!found || c < best) {
      found = true;
      best = c;
      std::memcpy(leh, ta, 16);
      std::memcpy(lel, tb, 16);
    }
  }
  return found;
}

void canonical_codes(const uint8_t* len, int n, uint32_t* code) {
  int bl_count[17] = {0};
  uint32_t next_code[17] = {0};
  for (int s = 0; s < n; ++s)
    if (len[s]) bl_count[len[s]]++;
  uint32_t c = 0;
  for (int bits = 1; bits <= 16; ++bits) {
    c = (c + (uint32_t)bl_count[bits - 1]) << 1;
    next_code[bits] = c;
  }
  for (int s = 0; s < n; ++s) code[s] = len[s] ? next_code[len[s]]++ : 0;
}

static uint32_t bit_reverse(uint32_t v, int n) {
  uint32_t r = 0;
  for (int i = 0; i < n; ++i) r = (r << 1) | ((v >> i) & 1u);
  return r;
}

// Checks lengths against the field's presence data: Kraft sum exactly one for
// two or more symbols, all zero for one symbol, every length <= lmax.
bool field_code_valid(const hl_field_code& fc, uint32_t lmax) {
  if (fc.nsym < 1 || fc.nsym > 16) return false;
  if (fc.nsym == 1) {
    if (fc.single > 15) return false;
    for (int s = 0; s < 16; ++s) if (fc.len[s]) return false;
    return true;
  }
  if (fc.single != 0) return false;
  int cnt = 0;
  uint64_t kraft = 0;  // in units of 2^-15
  for (int s = 0; s < 16; ++s) {
    if (!fc.len[s]) continue;
    if (fc.len[s] > lmax || fc.len[s] > 15) return false;
    ++cnt;
    kraft += 1ull << (15 - fc.len[s]);
  }
  return cnt == fc.nsym && kraft == (1ull << 15);
}

// Whole-exponent code: as above over 256 symbols, lengths <= lmax in [8, 13].
bool code8_valid(const hl_codebook8& cb) {
  if (cb.lmax < HL_LMAX8_MIN || cb.lmax > HL_LMAX8_MAX || cb.reserved) return false;
  if (cb.nsym < 1 || cb.nsym > 256) return false;
  if (cb.nsym == 1) {
    for (int s = 0; s < 256; ++s) if (cb.len[s]) return false;
    return true;
  }
  if (cb.single != 0) return false;
  int cnt = 0;
  uint64_t kraft = 0;  // in units of 2^-15
  for (int s = 0; s < 256; ++s) {
    if (!cb.len[s]) continue;
    if (cb.len[s] > cb.lmax) return false;
    ++cnt;
    kraft += 1ull << (15 - cb.len[s]);
  }
  return cnt == cb.nsym && kraft == (1ull << 15);
}

// One 5-bit field of the float16 format: as field_code_valid over 32 symbols.
static bool field5_valid(const hl_field_code5& fc, uint32_t lmax) {
  if (fc.nsym < 1 || fc.nsym > 32) return false;
  if (fc.nsym == 1) {
    if (fc.single > 31) return false;
    for (int s = 0; s < 32; ++s) if (fc.len[s]) return false;
    return true;
  }
  if (fc.single != 0) return false;
  int cnt = 0;
  uint64_t kraft = 0;  // in units of 2^-15
  for (int s = 0; s < 32; ++s) {
    if (!fc.len[s]) continue;
    if (fc.len[s] > lmax) return false;
    ++cnt;
    kraft += 1ull << (15 - fc.len[s]);
  }
  return cnt == fc.nsym && kraft == (1ull << 15);
}

bool code16_valid(const hl_codebook16& cb) {
  if (cb.lmax < HL_LMAX16_MIN || cb.lmax > HL_LMAX16_MAX) return false;
  return field5_valid(cb.e, cb.lmax) && field5_valid(cb.mh, cb.lmax) && field5_valid(cb.ml, cb.lmax);
}

// ---------------------------------------------------------------- layout

static uint64_t align64(uint64_t x) { return (x + 63) & ~uint64_t(63); }

bool shape_ok(uint64_t rows, uint64_t cols, uint32_t S) {
  return rows >= 1 && cols >= 1 && S >= 8 && S <= 512 && S % 8 == 0 && cols % S == 0 &&
         rows <= (1ull << 40) / cols;
}

bool grp_rows_ok(uint64_t cols, uint32_t S, uint32_t GR) {
  if (GR == 0 || GR > HL_GROUP_SEGS || (GR & (GR - 1))) return false;
  return S && (cols / S) % (HL_GROUP_SEGS / GR) == 0;
}

uint32_t default_grp_rows(uint64_t cols, uint32_t S) {
  for (uint32_t gc : {4u, 2u, 1u})
    if (S && (cols / S) % gc == 0) return HL_GROUP_SEGS / gc;
  return HL_GROUP_SEGS;
}

Layout make_layout(uint64_t rows, uint64_t cols, uint32_t S, uint32_t GR, uint32_t format) {
  Layout L;
  L.n = rows * cols;
  L.n_seg = L.n / S;
  L.L = cols / S;
  L.GR = GR;
  L.GC = HL_GROUP_SEGS / GR;
  L.n_grp = (rows + GR - 1) / GR * (L.L / L.GC);
  const uint64_t section = format == HL_FORMAT_WHOLE_EXPONENT ? HL_LEN8_BYTES
                           : format == HL_FORMAT_FP16        ? HL_CB16_BYTES
                                                             : 0;
  L.off_seg_bits = align64(HL_HEADER_BYTES + section);
  L.off_grp_off = align64(L.off_seg_bits + L.n_seg);               // one byte per segment
  L.off_stream = align64(L.off_grp_off + 4 * (2 * L.n_grp + 1));   // start and base per group, the end
  return L;
}

// Header of either format; in the whole-exponent format also the
// code-length section that follows it.
static void pack_header(uint8_t* h, uint64_t rows, uint64_t cols, uint32_t S, uint32_t format,
                        uint32_t lmax, const hl_codebook* cb, const hl_codebook8* cb8,
                        const hl_codebook16* cb16, const Layout& L, uint64_t off_raw, uint64_t total,
                        uint32_t max_units) {
  std::memset(h, 0, HL_HEADER_BYTES);
  auto put32 = [&](int o, uint32_t v) { std::memcpy(h + o, &v, 4); };
  auto put64 = [&](int o, uint64_t v) { std::memcpy(h + o, &v, 8); };
  put32(0, HL_MAGIC);
  uint16_t ver = HL_VERSION;
  std::memcpy(h + 4, &ver, 2);
  h[6] = (uint8_t)lmax;
  h[7] = (uint8_t)format;
  put64(8, rows);
  put64(16, cols);
  put32(24, S);
  put32(28, L.GR);
  put64(32, L.n_seg);
  put64(40, L.n_grp);
  put64(48, L.off_seg_bits);
  put64(56, L.off_grp_off);
  put64(64, L.off_stream);
  put64(72, off_raw);
  put64(80, total);
  put32(88, max_units);
  if (format == HL_FORMAT_WHOLE_EXPONENT) {
    std::memcpy(h + 92, &cb8->nsym, 2);
    h[94] = cb8->single;
    std::memcpy(h + HL_HEADER_BYTES, cb8->len, HL_LEN8_BYTES);
  } else if (format == HL_FORMAT_FP16) {
    uint8_t* sec = h + HL_HEADER_BYTES;
    std::memset(sec, 0, HL_CB16_BYTES);
    const hl_field_code5* f[3] = {&cb16->e, &cb16->mh, &cb16->ml};
    for (int k = 0; k < 3; ++k) {
      sec[34 * k] = f[k]->nsym;
      sec[34 * k + 1] = f[k]->single;
      std::memcpy(sec + 34 * k + 2, f[k]->len, 32);
    }
  } else {
    h[92] = cb->eh.nsym;
    h[93] = cb->el.nsym;
    h[94] = cb->eh.single;
    h[95] = cb->el.single;
    std::memcpy(h + 96, cb->eh.len, 16);
    std::memcpy(h + 112, cb->el.len, 16);
  }
}

bool parse_header(const uint8_t* h, size_t bytes, Header* o) {
  if (bytes < HL_HEADER_BYTES) return false;
  auto get32 = [&](int off) { uint32_t v; std::memcpy(&v, h + off, 4); return v; };
  auto get64 = [&](int off) { uint64_t v; std::memcpy(&v, h + off, 8); return v; };
  uint16_t ver;
  std::memcpy(&ver, h + 4, 2);
  if (get32(0) != HL_MAGIC || ver != HL_VERSION || h[7] > HL_FORMAT_FP16) return false;
  std::memset(o, 0, sizeof(*o));
  o->format = h[7];
  o->lmax = h[6];
  o->rows = get64(8);
  o->cols = get64(16);
  o->seg_len = get32(24);
  o->grp_rows = get32(28);
  o->n_seg = get64(32);
  o->n_grp = get64(40);
  o->off_seg_bits = get64(48);
  o->off_grp_off = get64(56);
  o->off_stream = get64(64);
  o->off_raw = get64(72);
  o->total_bytes = get64(80);
  o->max_grp_units = get32(88);
  if (o->format == HL_FORMAT_WHOLE_EXPONENT) {
    if (bytes < HL_HEADER_BYTES + HL_LEN8_BYTES) return false;
    for (int i = 95; i < (int)HL_HEADER_BYTES; ++i)
      if (h[i]) return false;
    o->cb8.lmax = o->lmax;
    std::memcpy(&o->cb8.nsym, h + 92, 2);
    o->cb8.single = h[94];
    std::memcpy(o->cb8.len, h + HL_HEADER_BYTES, HL_LEN8_BYTES);
  } else if (o->format == HL_FORMAT_FP16) {
    if (bytes < HL_HEADER_BYTES + HL_CB16_BYTES) return false;
    for (int i = 92; i < (int)HL_HEADER_BYTES; ++i)
      if (h[i]) return false;
    const uint8_t* sec = h + HL_HEADER_BYTES;
    for (int i = 102; i < (int)HL_CB16_BYTES; ++i)
      if (sec[i]) return false;
    o->cb16.lmax = o->lmax;
    hl_field_code5* f[3] = {&o->cb16.e, &o->cb16.mh, &o->cb16.ml};
    for (int k = 0; k < 3; ++k) {
      f[k]->nsym = sec[34 * k];
      f[k]->single = sec[34 * k + 1];
      std::memcpy(f[k]->len, sec + 34 * k + 2, 32);
    }
  } else {
    o->cb.lmax = o->lmax;
    o->cb.eh.nsym = h[92];
    o->cb.el.nsym = h[93];
    o->cb.eh.single = h[94];
    o->cb.el.single = h[95];
    std::memcpy(o->cb.eh.len, h + 96, 16);
    std::memcpy(o->cb.el.len, h + 112, 16);
  }
  return true;
}

// Longest code of one weight: a pair of field codes, or one exponent code.
static uint64_t weight_bits_max(const Header& H) {
  return H.format == HL_FORMAT_WHOLE_EXPONENT ? H.lmax : H.format == HL_FORMAT_FP16 ? 3ull * H.lmax : 2ull * H.lmax;
}

// Consistency of a parsed header with the layout rules (no data access).
bool header_consistent(const Header& H, uint64_t blob_bytes) {
  if (H.format == HL_FORMAT_WHOLE_EXPONENT) {
    if (!code8_valid(H.cb8)) return false;
  } else if (H.format == HL_FORMAT_FP16) {
    if (!code16_valid(H.cb16)) return false;
  } else {
    if (H.cb.lmax < 4 || H.cb.lmax > 15) return false;
    if (!field_code_valid(H.cb.eh, H.cb.lmax) || !field_code_valid(H.cb.el, H.cb.lmax)) return false;
  }
  if (!shape_ok(H.rows, H.cols, H.seg_len) || !grp_rows_ok(H.cols, H.seg_len, H.grp_rows)) return false;
  Layout L = make_layout(H.rows, H.cols, H.seg_len, H.grp_rows, H.format);
  if (H.n_seg != L.n_seg || H.n_grp != L.n_grp || H.off_seg_bits != L.off_seg_bits ||
      H.off_grp_off != L.off_grp_off || H.off_stream != L.off_stream)
    return false;
  if (H.off_raw < L.off_stream || H.off_raw % 64 || H.total_bytes != H.off_raw + raw_bytes(L.n, H.format))
    return false;
  if (H.total_bytes > blob_bytes) return false;
  // a group holds at most 64 * S weights of at most weight_bits_max bits
  uint64_t max_units = (64ull * H.seg_len * weight_bits_max(H) + 127) / 128;
  if (H.max_grp_units > max_units) return false;
  return true;
}

// Nearest (by ratio, the larger on a tie) to `target` among the multiples of
// 8 in [8, hi] that divide cols, restricted to cols/S % 4 == 0 if quad.
static uint32_t nearest_seg_len(uint64_t cols, uint32_t target, uint32_t hi, bool quad) {
  uint32_t best = 0;
  double bd = 1e30;
  for (uint32_t S = 8; S <= hi; S += 8) {
    if (cols % S || (quad && (cols / S) % 4)) continue;
    double d = S > target ? (double)S / target : (double)target / S;
    if (d <= bd + 1e-12) { bd = d; best = S; }
  }
  return best;
}

uint32_t default_seg_len(uint64_t cols) {
  const uint32_t S = nearest_seg_len(cols, 64, 128, true);
  return S ? S : nearest_seg_len(cols, 128, 512, false);
}

GroupGeom group_geom(uint64_t rows, uint64_t L, uint32_t GR, uint64_t g) {
  GroupGeom q;
  q.GC = HL_GROUP_SEGS / GR;
  const uint64_t CB = L / q.GC;
  const uint64_t rb = g / CB;
  q.c0 = (g % CB) * q.GC;
  q.r0 = rb * GR;
  q.G = (uint32_t)std::min<uint64_t>(GR, rows - q.r0);
  q.first = q.r0 * L + q.c0 * q.G;
  return q;
}

}  // namespace hl

using namespace hl;

// ---------------------------------------------------------------- C ABI

extern "C" const char* hl_status_str(hl_status s) {
  switch (s) {
    case HL_OK: return "ok";
    case HL_EINVAL: return "invalid argument";
    case HL_ENOMEM: return "buffer too small or out of host memory";
    case HL_ECORRUPT: return "corrupt container";
    case HL_EUNSUPPORTED: return "unsupported";
    case HL_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

extern "C" uint32_t hl_default_seg_len(uint64_t cols) { return default_seg_len(cols); }

// Threads for nthreads == 0: the CPUs this process may run on (its affinity
// mask, not the whole machine), at most 64.
static unsigned pick_threads(uint32_t nthreads) {
  unsigned t = nthreads;
  if (!t) {
    cpu_set_t set;
    t = sched_getaffinity(0, sizeof(set), &set) == 0 ? (unsigned)CPU_COUNT(&set)
                                                      : std::thread::hardware_concurrency();
  }
  return std::max(1u, std::min(t, 64u));
}

template <class F>
static void parallel_for(uint64_t n, unsigned nt, F f) {
  if (nt <= 1 || n < 2) { f(0, n); return; }
  std::vector<std::thread> th;
  uint64_t per = (n + nt - 1) / nt;
  for (unsigned t = 0; t < nt; ++t) {
    uint64_t a = t * per, b = std::min(n, a + per);
    if (a >= b) break;
    th.emplace_back([=] { f(a, b); });
  }
  for (auto& x : th) x.join();
}

// Histogram of the bits (v >> shift) & mask of n weights, over all cores for
// large inputs; nb = mask + 1 bins.
static std::vector<uint64_t> histogram(const uint16_t* w, size_t n, int shift, uint32_t mask) {
  const size_t nb = mask + 1;
  unsigned nt = pick_threads(0);
  if (n < (1u << 20)) nt = 1;
  const uint64_t per = (n + nt - 1) / nt;
  std::vector<std::vector<uint64_t>> part(nt, std::vector<uint64_t>(nb, 0));
  parallel_for(n, nt, [&](uint64_t a, uint64_t b) {
    std::vector<uint64_t>& h = part[a / per];
    for (uint64_t i = a; i < b; ++i) h[(w[i] >> shift) & mask]++;
  });
  std::vector<uint64_t> f(nb, 0);
  for (auto& h : part)
    for (size_t s = 0; s < nb; ++s) f[s] += h[s];
  return f;
}

extern "C" hl_status hl_build_codebook(const uint16_t* w, size_t n, uint32_t lmax, uint32_t pair_max,
                                       hl_codebook* out) {
  if (!w || !out || n == 0 || lmax < 4 || lmax > 15 || pair_max > 30) return HL_EINVAL;
  const std::vector<uint64_t> feh = histogram(w, n, 11, 15), fel = histogram(w, n, 7, 15);
  hl_codebook cb;
  std::memset(&cb, 0, sizeof(cb));
  cb.lmax = lmax;
  field_presence(feh.data(), &cb.eh);
  field_presence(fel.data(), &cb.el);
  if (!pair_limited_lengths(feh.data(), fel.data(), (int)lmax, (int)pair_max, cb.eh.len, cb.el.len))
    return HL_EINVAL;
  *out = cb;
  return HL_OK;
}

extern "C" hl_status hl_build_codebook8(const uint16_t* w, size_t n, uint32_t lmax, hl_codebook8* out) {
  if (!w || !out || n == 0 || lmax < HL_LMAX8_MIN || lmax > HL_LMAX8_MAX) return HL_EINVAL;
  const std::vector<uint64_t> f = histogram(w, n, 7, 255);
  std::memset(out, 0, sizeof(*out));
  out->lmax = lmax;
  int nsym = 0, single = 0;
  for (int s = 0; s < 256; ++s)
    if (f[s]) { ++nsym; single = s; }
  out->nsym = (uint16_t)nsym;
  out->single = (uint8_t)(nsym == 1 ? single : 0);
  limited_lengths(f.data(), 256, (int)lmax, out->len);
  return HL_OK;
}

extern "C" uint32_t hl_default_grp_rows(uint64_t cols, uint32_t seg_len) {
  return default_grp_rows(cols, seg_len ? seg_len : default_seg_len(cols));
}

// Code of each exponent byte e = (w >> 7) & 255 as it enters the stream: the
// bit-reversed code (LSB-first packing of an MSB-first code), its length, and
// whether e can be coded at all.
struct ByteCode {
  std::array<uint32_t, 256> code;
  std::array<uint8_t, 256> len;
  std::array<bool, 256> valid;
};

// Split format: the pair code(el) then code(eh).
static ByteCode pair_code(const hl_codebook& cb) {
  uint32_t ceh[16], cel[16];
  canonical_codes(cb.eh.len, 16, ceh);
  canonical_codes(cb.el.len, 16, cel);
  uint8_t leh[16], lel[16];
  bool veh[16], vel[16];
  for (int s = 0; s < 16; ++s) {
    leh[s] = cb.eh.nsym == 1 ? 0 : cb.eh.len[s];
    lel[s] = cb.el.nsym == 1 ? 0 : cb.el.len[s];
    veh[s] = cb.eh.nsym == 1 ? (s == cb.eh.single) : cb.eh.len[s] != 0;
    vel[s] = cb.el.nsym == 1 ? (s == cb.el.single) : cb.el.len[s] != 0;
  }
  ByteCode bc;
  for (int e = 0; e < 256; ++e) {
    int a = e >> 4, b = e & 15;
    bc.code[e] = bit_reverse(cel[b], lel[b]) | (bit_reverse(ceh[a], leh[a]) << lel[b]);
    bc.len[e] = (uint8_t)(leh[a] + lel[b]);
    bc.valid[e] = veh[a] && vel[b];
  }
  return bc;
}

// Whole-exponent format: one code per exponent byte.
static ByteCode whole_code(const hl_codebook8& cb) {
  uint32_t c[256];
  canonical_codes(cb.len, 256, c);
  ByteCode bc;
  for (int e = 0; e < 256; ++e) {
    bc.len[e] = cb.nsym == 1 ? 0 : cb.len[e];
    bc.code[e] = bit_reverse(c[e], bc.len[e]);
    bc.valid[e] = cb.nsym == 1 ? e == cb.single : cb.len[e] != 0;
  }
  return bc;
}

// Per-weight coders. len/valid/emit see a weight's 16 bits; emit passes its
// code parts, in stream order, to put(bit-reversed code, length).
// bf16 formats: the exponent byte's code (a pair, or one whole-exponent code),
// raw plane of (sign<<7 | mantissa) bytes.
struct ByteCoder {
  ByteCode bc;
  static constexpr bool kSignPlane = false;
  uint32_t len(uint32_t v) const { return bc.len[(v >> 7) & 0xFF]; }
  bool valid(uint32_t v) const { return bc.valid[(v >> 7) & 0xFF]; }
  template <class Put>
  void emit(uint32_t v, Put put) const {
    const uint32_t e = (v >> 7) & 0xFF;
    put(bc.code[e], bc.len[e]);
  }
};

// Float16 format: code(ml), code(e), code(mh); raw plane of sign bits.
struct F16Coder {
  uint32_t code[3][32];  // parts in stream order: ml, e, mh
  uint8_t plen[3][32];
  bool ok[3][32];
  static constexpr bool kSignPlane = true;
  static uint32_t part(uint32_t v, int k) { return k == 0 ? v & 31 : k == 1 ? (v >> 10) & 31 : (v >> 5) & 31; }
  explicit F16Coder(const hl_codebook16& cb) {
    const hl_field_code5* f[3] = {&cb.ml, &cb.e, &cb.mh};
    for (int k = 0; k < 3; ++k) {
      uint32_t c[32];
      canonical_codes(f[k]->len, 32, c);
      for (int s = 0; s < 32; ++s) {
        plen[k][s] = f[k]->nsym == 1 ? 0 : f[k]->len[s];
        code[k][s] = bit_reverse(c[s], plen[k][s]);
        ok[k][s] = f[k]->nsym == 1 ? s == f[k]->single : f[k]->len[s] != 0;
      }
    }
  }
  uint32_t len(uint32_t v) const { return plen[0][part(v, 0)] + plen[1][part(v, 1)] + plen[2][part(v, 2)]; }
  bool valid(uint32_t v) const { return ok[0][part(v, 0)] && ok[1][part(v, 1)] && ok[2][part(v, 2)]; }
  template <class Put>
  void emit(uint32_t v, Put put) const {
    for (int k = 0; k < 3; ++k) put(code[k][part(v, k)], plen[k][part(v, k)]);
  }
};

// The encoder proper, shared by all formats: everything but the header, the
// per-weight coder and the raw plane's kind is format independent.
template <class Coder>
static hl_status encode_body(const uint16_t* w, uint64_t rows, uint64_t cols, uint32_t seg_len,
                             uint32_t grp_rows, uint32_t nthreads, uint32_t format, uint32_t lmax,
                             const hl_codebook* cb, const hl_codebook8* cb8, const hl_codebook16* cb16,
                             const Coder& cd, void* out, size_t* out_bytes) {
  const uint32_t S = seg_len;
  const uint32_t GR = grp_rows;
  Layout L = make_layout(rows, cols, S, GR, format);
  const unsigned nt = pick_threads(nthreads);
  // Pass 1: segment bit counts, in group order.
  std::vector<uint16_t> seg_bits(L.n_seg);
  std::vector<uint8_t> bad(nt, 0);
  const uint64_t per1 = (L.n_grp + nt - 1) / nt;
  parallel_for(L.n_grp, nt, [&](uint64_t a, uint64_t b) {
    bool anybad = false;
    for (uint64_t g = a; g < b; ++g) {
      GroupGeom q = group_geom(rows, L.L, GR, g);
      for (uint32_t mu = 0; mu < q.G * q.GC; ++mu) {
        const uint16_t* p = w + (q.r0 + mu % q.G) * cols + (q.c0 + mu / q.G) * S;
        uint32_t bits = 0;
        for (uint32_t t = 0; t < S; ++t) {
          anybad |= !cd.valid(p[t]);
          bits += cd.len(p[t]);
        }
        seg_bits[q.first + mu] = (uint16_t)bits;
      }
    }
    if (anybad) bad[a / per1] = 1;
  });
  for (auto b : bad)
    if (b) return HL_EINVAL;
  // Stored segment lengths: the group's base (its least code-bit count, or
  // its greatest minus 255 when they span more) plus one byte per segment,
  // shorter segments padded to base with zero bits. Group stream sizes
  // (16-byte units), starts and bases.
  std::vector<uint8_t> seg_len8(L.n_seg);
  std::vector<uint32_t> grp_meta(2 * L.n_grp + 1);
  uint64_t units = 0;
  uint32_t max_units = 0;
  for (uint64_t g = 0; g < L.n_grp; ++g) {
    GroupGeom q = group_geom(rows, L.L, GR, g);
    const uint32_t NG = q.G * q.GC;
    uint32_t lo = 0xFFFFFFFFu, hi = 0;
    for (uint32_t mu = 0; mu < NG; ++mu) {
      lo = std::min<uint32_t>(lo, seg_bits[q.first + mu]);
      hi = std::max<uint32_t>(hi, seg_bits[q.first + mu]);
    }
    const uint32_t base = hi > lo + kSegLenSpan ? hi - kSegLenSpan : lo;
    uint64_t bits = 0;
    for (uint32_t mu = 0; mu < NG; ++mu) {
      const uint32_t stored = std::max<uint32_t>(seg_bits[q.first + mu], base);
      seg_len8[q.first + mu] = (uint8_t)(stored - base);
      bits += stored;
    }
    uint64_t u = (bits + 127) / 128;
    grp_meta[2 * g] = (uint32_t)units;
    grp_meta[2 * g + 1] = base;
    units += u;
    max_units = std::max<uint32_t>(max_units, (uint32_t)u);
    if (units > 0xFFFFFFFFull) return HL_EUNSUPPORTED;
  }
  grp_meta[2 * L.n_grp] = (uint32_t)units;
  const uint64_t off_raw = align64(L.off_stream + units * 16);
  const uint64_t total = off_raw + raw_bytes(L.n, format);
  if (!out) { *out_bytes = total; return HL_OK; }
  if (*out_bytes < total) { *out_bytes = total; return HL_ENOMEM; }
  uint8_t* o = (uint8_t*)out;
  std::memset(o, 0, L.off_stream);  // header, codebook section, padding, metadata
  pack_header(o, rows, cols, S, format, lmax, cb, cb8, cb16, L, off_raw, total, max_units);
  std::memcpy(o + L.off_seg_bits, seg_len8.data(), L.n_seg);
  std::memcpy(o + L.off_grp_off, grp_meta.data(), 4 * (2 * L.n_grp + 1));
  std::memset(o + L.off_stream + units * 16, 0, off_raw - (L.off_stream + units * 16));
  // Pass 2: group streams and raw plane, independent per group.
  parallel_for(L.n_grp, nt, [&](uint64_t ga, uint64_t gb) {
    for (uint64_t g = ga; g < gb; ++g) {
      GroupGeom q = group_geom(rows, L.L, GR, g);
      uint32_t* dst = (uint32_t*)(o + L.off_stream + (uint64_t)grp_meta[2 * g] * 16);
      const uint64_t nwords = (uint64_t)(grp_meta[2 * g + 2] - grp_meta[2 * g]) * 4;
      const uint32_t base = grp_meta[2 * g + 1];
      uint64_t acc = 0;
      int nb = 0;
      uint64_t wi = 0;
      // each part is at most 16 bits and nb < 32 before it: acc never overflows
      auto put = [&](uint32_t code, uint32_t len) {
        acc |= (uint64_t)code << nb;
        nb += (int)len;
        if (nb >= 32) {
          dst[wi++] = (uint32_t)acc;
          acc >>= 32;
          nb -= 32;
        }
      };
      const uint32_t NG = q.G * q.GC;
      for (uint32_t mu = 0; mu < NG; ++mu) {
        const uint16_t* p = w + (q.r0 + mu % q.G) * cols + (q.c0 + mu / q.G) * S;
        if (Coder::kSignPlane) {
          // sign bits: byte (segment number)*S/8 + t/8, bit t%8
          uint8_t* sdst = o + off_raw + (q.first + mu) * (S / 8);
          for (uint32_t t = 0; t < S; t += 8) {
            uint32_t byte = 0;
            for (uint32_t k = 0; k < 8; ++k) {
              cd.emit(p[t + k], put);
              byte |= (uint32_t)(p[t + k] >> 15) << k;
            }
            sdst[t / 8] = (uint8_t)byte;
          }
        } else {
          // raw plane: ((t/8)*NG + mu)*8 + t%8 within the group
          uint8_t* rdst = o + off_raw + q.first * S;
          for (uint32_t t = 0; t < S; ++t) {
            const uint32_t v = p[t];
            cd.emit(v, put);
            rdst[((t >> 3) * NG + mu) * 8 + (t & 7)] = (uint8_t)(((v >> 8) & 0x80) | (v & 0x7F));
          }
        }
        // a segment shorter than the group's base: zero bits up to it
        for (uint32_t pad = base > seg_bits[q.first + mu] ? base - seg_bits[q.first + mu] : 0; pad;) {
          const uint32_t k = std::min<uint32_t>(pad, 16);
          put(0, k);
          pad -= k;
        }
      }
      while (wi < nwords) {  // tail bits, then zero padding to 128 bits
        dst[wi++] = (uint32_t)acc;
        acc >>= 32;
      }
    }
  });
  *out_bytes = total;
  return HL_OK;
}

// Shape arguments of both encoders: the segment length and group rows used.
static bool resolve_shape(uint64_t rows, uint64_t cols, uint32_t seg_len, uint32_t grp_rows, uint32_t* S,
                          uint32_t* GR) {
  *S = seg_len ? seg_len : default_seg_len(cols);
  if (!shape_ok(rows, cols, *S)) return false;
  *GR = grp_rows ? grp_rows : default_grp_rows(cols, *S);
  return grp_rows_ok(cols, *S, *GR);
}

extern "C" hl_status hl_encode(const uint16_t* w, uint64_t rows, uint64_t cols, const hl_codebook* cb,
                               uint32_t seg_len, uint32_t grp_rows, uint32_t nthreads, void* out,
                               size_t* out_bytes) {
  if (!w || !cb || !out_bytes) return HL_EINVAL;
  uint32_t S, GR;
  if (!resolve_shape(rows, cols, seg_len, grp_rows, &S, &GR)) return HL_EINVAL;
  if (cb->lmax < 4 || cb->lmax > 15 || !field_code_valid(cb->eh, cb->lmax) ||
      !field_code_valid(cb->el, cb->lmax))
    return HL_EINVAL;
  return encode_body(w, rows, cols, S, GR, nthreads, HL_FORMAT_SPLIT, cb->lmax, cb, nullptr, nullptr,
                     ByteCoder{pair_code(*cb)}, out, out_bytes);
}

extern "C" hl_status hl_encode8(const uint16_t* w, uint64_t rows, uint64_t cols, const hl_codebook8* cb,
                                uint32_t seg_len, uint32_t grp_rows, uint32_t nthreads, void* out,
                                size_t* out_bytes) {
  if (!w || !cb || !out_bytes) return HL_EINVAL;
  uint32_t S, GR;
  if (!resolve_shape(rows, cols, seg_len, grp_rows, &S, &GR)) return HL_EINVAL;
  if (!code8_valid(*cb)) return HL_EINVAL;
  return encode_body(w, rows, cols, S, GR, nthreads, HL_FORMAT_WHOLE_EXPONENT, cb->lmax, nullptr, cb, nullptr,
                     ByteCoder{whole_code(*cb)}, out, out_bytes);
}

extern "C" hl_status hl_build_codebook16(const uint16_t* w, size_t n, uint32_t lmax, hl_codebook16* out) {
  if (!w || !out || n == 0 || lmax < HL_LMAX16_MIN || lmax > HL_LMAX16_MAX) return HL_EINVAL;
  std::memset(out, 0, sizeof(*out));
  out->lmax = lmax;
  const int shift[3] = {10, 5, 0};
  hl_field_code5* f[3] = {&out->e, &out->mh, &out->ml};
  for (int k = 0; k < 3; ++k) {
    const std::vector<uint64_t> h = histogram(w, n, shift[k], 31);
    int nsym = 0, single = 0;
    for (int s = 0; s < 32; ++s)
      if (h[s]) { ++nsym; single = s; }
    f[k]->nsym = (uint8_t)nsym;
    f[k]->single = (uint8_t)(nsym == 1 ? single : 0);
    limited_lengths(h.data(), 32, (int)lmax, f[k]->len);
  }
  return HL_OK;
}

extern "C" hl_status hl_encode16(const uint16_t* w, uint64_t rows, uint64_t cols, const hl_codebook16* cb,
                                 uint32_t seg_len, uint32_t grp_rows, uint32_t nthreads, void* out,
                                 size_t* out_bytes) {
  if (!w || !cb || !out_bytes) return HL_EINVAL;
  uint32_t S, GR;
  if (!resolve_shape(rows, cols, seg_len, grp_rows, &S, &GR)) return HL_EINVAL;
  if (!code16_valid(*cb)) return HL_EINVAL;
  return encode_body(w, rows, cols, S, GR, nthreads, HL_FORMAT_FP16, cb->lmax, nullptr, nullptr, cb,
                     F16Coder(*cb), out, out_bytes);
}

namespace hl {

hl_status validate_blob(const uint8_t* b, size_t bytes, Header* out, uint32_t* max_seg_bits) {
  if (!b || bytes < HL_HEADER_BYTES) return HL_ECORRUPT;
  Header H;
  if (!parse_header(b, bytes, &H) || !header_consistent(H, bytes)) return HL_ECORRUPT;
  const uint8_t* sb = b + H.off_seg_bits;                             // one byte per segment
  const uint32_t* gm = (const uint32_t*)(b + H.off_grp_off);          // start, base per group; end
  if (gm[0] != 0) return HL_ECORRUPT;
  uint32_t mx = 0, mseg = 0;
  const uint64_t max_seg = (uint64_t)H.seg_len * weight_bits_max(H);
  const uint64_t L = H.cols / H.seg_len;
  for (uint64_t g = 0; g < H.n_grp; ++g) {
    GroupGeom q = group_geom(H.rows, L, H.grp_rows, g);
    const uint32_t base = gm[2 * g + 1];
    uint64_t bits = 0;
    for (uint32_t mu = 0; mu < q.G * q.GC; ++mu) {
      const uint64_t v = (uint64_t)base + sb[q.first + mu];
      if (v > max_seg) return HL_ECORRUPT;
      bits += v;
      mseg = std::max(mseg, (uint32_t)v);
    }
    const uint32_t u0 = gm[2 * g], u1 = gm[2 * g + 2];
    if (u1 < u0 || u1 - u0 != (bits + 127) / 128) return HL_ECORRUPT;
    mx = std::max(mx, u1 - u0);
  }
  if (mx != H.max_grp_units) return HL_ECORRUPT;
  if (H.off_raw != align64(H.off_stream + (uint64_t)gm[2 * H.n_grp] * 16)) return HL_ECORRUPT;
  if (out) *out = H;
  if (max_seg_bits) *max_seg_bits = mseg;
  return HL_OK;
}

}  // namespace hl

extern "C" hl_status hl_validate(const void* blob, size_t bytes) {
  return validate_blob((const uint8_t*)blob, bytes, nullptr, nullptr);
}
