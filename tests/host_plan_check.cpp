// Host-only check of the planner and validators (plan.cpp), built with g++ and the address and
// undefined-behaviour sanitizers by tests/test_host_sanitizers.py.  It runs randomized decode and prefill
// plans (lengths 0..200k tokens, empty sequences, groups of 1..80 members, GQA ratios 1..16) and checks
// every property the kernels rely on:
//   decode:  each (sequence, page) pair is read exactly once for its query columns (a shared page once
//            for every member of the unit that reads it), token ends match the sequence lengths, every
//            partial slot of a sequence is written exactly once, segments never exceed the split size
//            (pages plus a start cost per chunk) and fit one round of waves;
//   prefill: every (session, KV head, query row) is covered exactly once per key range, the key ranges
//            of a tile tile [0, its last key] without gaps or overlaps;
//            a split call, and any call of at most one round, keeps every XCD within its share of the
//            resident workgroups;
//   both:    plans are deterministic, and invalid inputs return the documented error codes.
// `self-test` plants mistakes into plans and expects the checks to reject each of them.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <random>
#include <string>
#include <vector>

#include "../paper_2608_11152_amd/csrc/kvp_plan.h"

using kvp::DecodeItem;
using kvp::DecodePlan;
using kvp::PrefillItem;
using kvp::PrefillPlan;

static int g_fail = 0;
#define EXPECT(c, ...)                                  \
  do {                                                  \
    if (!(c)) {                                         \
      std::fprintf(stderr, "check failed: " __VA_ARGS__); \
      std::fprintf(stderr, "\n");                       \
      return false;                                     \
    }                                                   \
  } while (0)

struct DecodeCase {
  std::vector<int32_t> lens, gid, shared;
  int Hq = 32, Hkv = 4, maxp = 0;
};

static bool check_decode(const DecodeCase& c, const DecodePlan& P, int K = kvp::kChunkStartPages) {
  const int B = (int)c.lens.size();
  std::vector<std::vector<int>> seen(B);
  for (int i = 0; i < B; ++i) seen[i].assign((c.lens[i] + 15) / 16, 0);
  std::vector<std::vector<int>> slot_seen(B);
  for (int i = 0; i < B; ++i) slot_seen[i].assign(P.n_parts[i] > 0 ? P.n_parts[i] : 0, 0);
  const int G = c.Hq / c.Hkv;
  auto visit = [&](const DecodeItem& it, bool wave) -> bool {
    EXPECT(it.page_lo >= 0 && it.page_lo < it.page_hi, "item page range [%d, %d)", it.page_lo, it.page_hi);
    EXPECT(it.n_mem >= 1 && it.mem_off >= 0 && it.mem_off + it.n_mem <= (int)P.members.size(), "member list");
    EXPECT(it.n_mem * G <= (wave ? kvp::kMaxColsPerWave : kvp::kMaxColsPerGroup), "%d columns on the %s path",
           it.n_mem * G, wave ? "wave" : "group");
    EXPECT(wave || it.n_mem * G > kvp::kMaxColsPerWave, "a narrow unit on the group path");
    const int row = it.row;
    EXPECT(row >= 0 && row < B, "row %d", row);
    if (it.kind == 0) {
      EXPECT(it.n_mem == 1 && P.members[it.mem_off] == row, "private item owner");
      EXPECT(it.tok_end == c.lens[row], "private token end %d vs len %d", it.tok_end, c.lens[row]);
    } else {
      EXPECT(c.gid[row] >= 0, "prefix item of an ungrouped row");
      const int S = c.shared[c.gid[row]];
      EXPECT(it.page_hi <= S && it.tok_end == S * 16, "prefix range beyond the shared pages");
      EXPECT(P.members[it.mem_off] == row, "the representative is the unit's first member");
    }
    for (int m = 0; m < it.n_mem; ++m) {
      const int s = P.members[it.mem_off + m];
      EXPECT(s >= 0 && s < B && c.lens[s] > 0, "member %d", s);
      if (it.kind == 1) EXPECT(c.gid[s] == c.gid[row], "member of another group");
      for (int p = it.page_lo; p < it.page_hi; ++p) {
        EXPECT(p < (int)seen[s].size(), "page %d beyond sequence %d", p, s);
        seen[s][p]++;
      }
      if (it.slot >= 0) {
        EXPECT(it.slot < (int)slot_seen[s].size(), "slot %d of %d", it.slot, (int)slot_seen[s].size());
        slot_seen[s][it.slot]++;
      } else {
        EXPECT(P.n_parts[s] == 1, "a direct write for a merged sequence");
      }
    }
    return true;
  };
  EXPECT(P.seg_off.size() >= 1 && P.seg_off.front() == 0 && P.seg_off.back() == (int)P.wave_items.size(),
         "segment offsets");
  for (size_t s = 0; s + 1 < P.seg_off.size(); ++s) {
    EXPECT(P.seg_off[s] < P.seg_off[s + 1], "empty segment %zu", s);
    int pages = 0;
    for (int k = P.seg_off[s]; k < P.seg_off[s + 1]; ++k) pages += P.wave_items[k].page_hi - P.wave_items[k].page_lo;
    EXPECT(pages <= P.pages_per_split, "segment of %d pages > %d", pages, P.pages_per_split);
    // a segment's cost counts every chunk start as K pages; it stays within the budget
    const int cost = pages + K * (P.seg_off[s + 1] - P.seg_off[s]);
    EXPECT(cost <= P.pages_per_split + K, "segment cost %d > %d", cost, P.pages_per_split + K);
  }
  // one round of waves: every segment is taken by Hkv waves of the kDecodeWaves budget
  EXPECT((int64_t)(P.seg_off.size() - 1) * c.Hkv <= kvp::kDecodeWaves, "%zu segments x %d KV heads > %d waves",
         P.seg_off.size() - 1, c.Hkv, kvp::kDecodeWaves);
  for (const auto& it : P.wave_items)
    if (!visit(it, true)) return false;
  for (const auto& it : P.group_items)
    if (!visit(it, false)) return false;
  int32_t total = 0;
  for (int i = 0; i < B; ++i) {
    for (size_t p = 0; p < seen[i].size(); ++p) EXPECT(seen[i][p] == 1, "sequence %d page %zu read %d times", i, p, seen[i][p]);
    const bool merged = std::find(P.merge_seqs.begin(), P.merge_seqs.end(), i) != P.merge_seqs.end();
    if (c.lens[i] == 0) EXPECT(merged, "an empty sequence must get its zero output from the merge");
    if (merged) {
      EXPECT(P.part_base[i] == total, "partial base of sequence %d", i);
      total += P.n_parts[i];
      for (size_t k = 0; k < slot_seen[i].size(); ++k) EXPECT(slot_seen[i][k] == 1, "sequence %d slot %zu", i, k);
    } else {
      EXPECT(P.n_parts[i] == 1 && c.lens[i] > 0, "direct sequence %d", i);
    }
  }
  EXPECT(total == P.total_parts, "partial count %d vs %d", total, P.total_parts);
  return true;
}

struct PrefillCase {
  std::vector<int32_t> ctx, cuq;
  int Hq = 32, Hkv = 4, maxp = 0;
};

static bool check_prefill(const PrefillCase& c, const PrefillPlan& P) {
  const int B = (int)c.ctx.size();
  const int G = c.Hq / c.Hkv;
  // per (session, kv head, tile): the key stages covered, in order
  std::map<std::vector<int>, std::vector<std::pair<int, int>>> ranges;
  int64_t real = 0;
  for (const auto& it : P.items) {
    if (it.seq < 0) continue;
    ++real;
    EXPECT(it.seq < B && it.kvh >= 0 && it.kvh < c.Hkv, "item seq %d kvh %d", it.seq, it.kvh);
    const int C = c.cuq[it.seq + 1] - c.cuq[it.seq];
    EXPECT(it.row0 % kvp::kPrefillRows == 0 && it.row0 < C * G, "tile row %d of %d", it.row0, C * G);
    ranges[{it.seq, it.kvh, it.row0}].push_back({it.st_lo, it.st_hi});
    if (it.slot >= 0) EXPECT(it.st_hi > it.st_lo, "empty split");
  }
  EXPECT(real == P.real_items, "real items %lld vs %lld", (long long)real, (long long)P.real_items);
  {
    // A split history is cut into few enough ranges that the whole call is one round of the resident
    // workgroups, and a call that fits one round keeps every XCD (workgroup b on XCD b % 8) within its
    // share of them: the padded grid is at most kPrefillSplitTarget long.
    bool split = false;
    for (int32_t n : P.nsplit) split |= n > 1;
    if (split) EXPECT(P.real_items <= kvp::kPrefillSplitTarget, "split call of %lld workgroups", (long long)P.real_items);
    if (P.real_items <= kvp::kPrefillSplitTarget)
      EXPECT(P.items.size() <= (size_t)kvp::kPrefillSplitTarget, "one-round call padded to %zu workgroups",
             P.items.size());
  }
  {
    // every query row of a split session has nsplit partials of its own, in one merge record
    int32_t parts = 0;
    size_t rec = 0;
    for (int i = 0; i < B; ++i) {
      if (P.nsplit[i] == 1) continue;
      EXPECT(P.part_base[i] == parts, "partial base of session %d", i);
      for (int j = c.cuq[i]; j < c.cuq[i + 1]; ++j, ++rec) {
        EXPECT(4 * rec + 3 < P.merge_info.size(), "merge records");
        EXPECT(P.merge_info[4 * rec] == j && P.merge_info[4 * rec + 1] == parts + (j - c.cuq[i]) * P.nsplit[i] &&
                   P.merge_info[4 * rec + 2] == P.nsplit[i],
               "merge record of row %d", j);
      }
      parts += (c.cuq[i + 1] - c.cuq[i]) * P.nsplit[i];
    }
    EXPECT(4 * rec == P.merge_info.size() && parts == P.total_parts, "merge records and partial count");
    for (const auto& it : P.items)
      if (it.seq >= 0) EXPECT((it.slot >= 0) == (P.nsplit[it.seq] > 1) && it.slot < P.nsplit[it.seq], "slot");
  }
  for (int i = 0; i < B; ++i) {
    const int C = c.cuq[i + 1] - c.cuq[i];
    const int nt = (C * G + kvp::kPrefillRows - 1) / kvp::kPrefillRows;
    for (int h = 0; h < c.Hkv; ++h)
      for (int t = 0; t < nt; ++t) {
        auto f = ranges.find({i, h, t * kvp::kPrefillRows});
        EXPECT(f != ranges.end(), "session %d head %d tile %d not covered", i, h, t);
        auto v = f->second;
        std::sort(v.begin(), v.end());
        const int last_row = std::min(C * G - 1, t * kvp::kPrefillRows + kvp::kPrefillRows - 1);
        const int n_keys = c.ctx[i] + last_row / G + 1;
        const int n_st = (n_keys + 63) / 64;
        int at = 0;
        for (auto& r : v) {
          EXPECT(r.first == at, "session %d tile %d: key stages start at %d, expected %d", i, t, r.first, at);
          // every query row sees the first key of every range (rows sit at positions >= ctx)
          EXPECT((int64_t)r.first * 64 <= c.ctx[i], "a range starts past the cached history");
          at = r.second;
        }
        EXPECT(at == n_st, "session %d tile %d: key stages end at %d of %d", i, t, at, n_st);
        EXPECT((int)v.size() == P.nsplit[i], "session %d: %zu ranges, nsplit %d", i, v.size(), P.nsplit[i]);
      }
  }
  return true;
}

static std::mt19937_64 rng;
static int uni(int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); }

static DecodeCase random_decode() {
  DecodeCase c;
  static const int Gs[] = {1, 2, 4, 8, 16};
  static const int Hkvs[] = {1, 2, 4, 8};
  const int G = Gs[uni(0, 4)];
  c.Hkv = Hkvs[uni(0, 3)];
  c.Hq = G * c.Hkv;
  const int n_groups = uni(0, 6);
  for (int g = 0; g < n_groups; ++g) {
    const int members = uni(0, 4) == 0 ? uni(20, 80) : uni(1, 12);
    const int S = uni(0, 3) == 0 ? 0 : uni(1, uni(0, 1) ? 64 : 2000);
    c.shared.push_back(S);
    for (int m = 0; m < members; ++m) {
      c.gid.push_back(g);
      const int priv = uni(0, 5) == 0 ? 0 : uni(1, uni(0, 3) == 0 ? 200000 - S * 16 : 5000);
      c.lens.push_back(uni(0, 9) == 0 && S == 0 ? 0 : S * 16 + priv);
    }
  }
  const int lone = uni(0, 40);
  for (int i = 0; i < lone; ++i) {
    c.gid.push_back(-1);
    c.lens.push_back(uni(0, 6) == 0 ? 0 : uni(1, uni(0, 4) == 0 ? 200000 : 3000));
  }
  for (int32_t n : c.lens) c.maxp = std::max(c.maxp, (n + 15) / 16);
  c.maxp += uni(0, 3);
  return c;
}

static PrefillCase random_prefill() {
  PrefillCase c;
  static const int Gs[] = {1, 2, 4, 8, 16};
  const int G = Gs[uni(0, 4)];
  c.Hkv = 1 << uni(0, 3);
  c.Hq = G * c.Hkv;
  const int B = uni(1, 12);
  c.cuq.push_back(0);
  for (int i = 0; i < B; ++i) {
    c.ctx.push_back(uni(0, 3) == 0 ? uni(0, 100) : uni(0, 200000));
    const int C = uni(0, 5) == 0 ? uni(0, 3) : uni(1, uni(0, 1) ? 300 : 2048);
    c.cuq.push_back(c.cuq.back() + C);
    c.maxp = std::max(c.maxp, (c.ctx.back() + C + 15) / 16);
  }
  return c;
}

static kvp_group_prefix gp_of(const DecodeCase& c) {
  kvp_group_prefix gp{c.gid.data(), c.shared.empty() ? nullptr : c.shared.data(), (int32_t)c.shared.size()};
  return gp;
}

static bool same_plan(const DecodePlan& a, const DecodePlan& b) {
  auto eq = [](const auto& x, const auto& y) {
    return x.size() == y.size() && (x.empty() || !std::memcmp(x.data(), y.data(), x.size() * sizeof(x[0])));
  };
  return eq(a.wave_items, b.wave_items) && eq(a.group_items, b.group_items) && eq(a.members, b.members) &&
         eq(a.seg_off, b.seg_off) && eq(a.part_base, b.part_base) && a.total_parts == b.total_parts;
}

static bool run_decode(const DecodeCase& c) {
  kvp_group_prefix gp = gp_of(c);
  DecodePlan P, Q;
  kvp::Status s = kvp::plan_decode(c.lens.data(), (int)c.lens.size(), c.maxp, &gp, c.Hq, c.Hkv, &P);
  EXPECT(s.ok(), "plan_decode failed: %s", s.msg.c_str());
  kvp::plan_decode(c.lens.data(), (int)c.lens.size(), c.maxp, &gp, c.Hq, c.Hkv, &Q);
  EXPECT(same_plan(P, Q), "plan_decode is not deterministic");
  if (!check_decode(c, P)) return false;
  // the FP8-pool plan: the same properties under its larger chunk-start cost
  DecodePlan F;
  s = kvp::plan_decode(c.lens.data(), (int)c.lens.size(), c.maxp, &gp, c.Hq, c.Hkv, &F, kvp::kChunkStartPagesFp8);
  EXPECT(s.ok(), "plan_decode (FP8 cost) failed: %s", s.msg.c_str());
  return check_decode(c, F, kvp::kChunkStartPagesFp8);
}

static int g_split_sessions = 0;

static bool run_prefill(const PrefillCase& c) {
  PrefillPlan P, Q;
  kvp::Status s = kvp::plan_prefill(c.ctx.data(), c.cuq.data(), (int)c.ctx.size(), c.maxp, c.Hq, c.Hkv, &P);
  EXPECT(s.ok(), "plan_prefill failed: %s", s.msg.c_str());
  for (int32_t n : P.nsplit) g_split_sessions += n > 1;
  kvp::plan_prefill(c.ctx.data(), c.cuq.data(), (int)c.ctx.size(), c.maxp, c.Hq, c.Hkv, &Q);
  EXPECT(P.items.size() == Q.items.size() &&
             (P.items.empty() || !std::memcmp(P.items.data(), Q.items.data(), P.items.size() * sizeof(PrefillItem))),
         "plan_prefill is not deterministic");
  return check_prefill(c, P);
}

static bool run_errors() {
  DecodeCase c;
  c.lens = {40, 50};
  c.gid = {0, 0};
  c.shared = {2};
  c.maxp = 4;
  kvp_group_prefix gp = gp_of(c);
  DecodePlan P;
  auto code = [&](const DecodeCase& x, int Hq, int Hkv) {
    kvp_group_prefix g = gp_of(x);
    return kvp::plan_decode(x.lens.data(), (int)x.lens.size(), x.maxp, &g, Hq, Hkv, &P).code;
  };
  EXPECT(code(c, 32, 4) == KVP_OK, "valid case");
  EXPECT(code(c, 24, 4) == KVP_EUNSUPPORTED, "GQA ratio 6");
  EXPECT(code(c, 30, 4) == KVP_EUNSUPPORTED, "Hq not a multiple of Hkv");
  DecodeCase d = c;
  d.lens[1] = 65;
  EXPECT(code(d, 32, 4) == KVP_ERANGE, "length beyond maxp * 16");
  d = c;
  d.lens[0] = -1;
  EXPECT(code(d, 32, 4) == KVP_EINVAL, "negative length");
  d = c;
  d.gid[1] = 1;
  EXPECT(code(d, 32, 4) == KVP_EGROUP, "group id out of range");
  d = c;
  d.shared[0] = 3;
  EXPECT(code(d, 32, 4) == KVP_EGROUP, "shared prefix longer than a member");
  d = c;
  d.shared[0] = -1;
  EXPECT(code(d, 32, 4) == KVP_EGROUP, "negative shared pages");
  EXPECT(kvp::plan_decode(c.lens.data(), -1, c.maxp, &gp, 32, 4, &P).code == KVP_EINVAL, "negative count");
  // tables: valid, an id outside the pool, a member whose shared entries differ
  std::vector<int32_t> bt = {0, 1, 2, -1, 0, 1, 3, 4};
  EXPECT(kvp::check_tables(bt.data(), 4, c.lens.data(), 2, 5, &gp).code == KVP_OK, "valid tables");
  EXPECT(kvp::check_tables(bt.data(), 4, c.lens.data(), 2, 4, &gp).code == KVP_ERANGE, "id outside the pool");
  bt[5] = 4;
  EXPECT(kvp::check_tables(bt.data(), 4, c.lens.data(), 2, 5, &gp).code == KVP_EGROUP, "members differ");
  PrefillPlan Q;
  std::vector<int32_t> ctx = {10, 20}, cuq = {0, 5, 9};
  EXPECT(kvp::plan_prefill(ctx.data(), cuq.data(), 2, 2, 32, 4, &Q).code == KVP_OK, "valid prefill");
  EXPECT(kvp::plan_prefill(ctx.data(), cuq.data(), 2, 1, 32, 4, &Q).code == KVP_ERANGE, "prefill beyond maxp");
  cuq[1] = 10;
  EXPECT(kvp::plan_prefill(ctx.data(), cuq.data(), 2, 2, 32, 4, &Q).code == KVP_EINVAL, "cu_q decreases");
  return true;
}

// Planted mistakes: each corrupted plan must be rejected by the checks above.
static bool self_test() {
  rng.seed(7);
  DecodeCase c;
  do c = random_decode(); while (c.shared.empty() || c.lens.size() < 4);
  kvp_group_prefix gp = gp_of(c);
  DecodePlan P;
  kvp::plan_decode(c.lens.data(), (int)c.lens.size(), c.maxp, &gp, c.Hq, c.Hkv, &P);
  int rejected = 0, planted = 0;
  auto expect_reject = [&](DecodePlan bad) {
    ++planted;
    if (!check_decode(c, bad)) ++rejected;
  };
  if (!P.wave_items.empty()) {
    DecodePlan b = P;
    b.wave_items.back().page_hi -= 1;  // a page never read
    if (b.wave_items.back().page_hi > b.wave_items.back().page_lo) expect_reject(b);
    b = P;
    b.wave_items.push_back(P.wave_items.back());  // a chunk read twice
    b.seg_off.back() += 1;
    expect_reject(b);
    b = P;
    b.wave_items[0].tok_end += 1;  // wrong token end
    expect_reject(b);
    if (P.seg_off.size() > 2) {
      b = P;
      b.seg_off.erase(b.seg_off.begin() + 1);  // two segments given to one wave
      expect_reject(b);
    }
  }
  {
    DecodePlan b = P;
    b.total_parts += 1;
    expect_reject(b);
  }
  PrefillCase pc;
  pc.ctx = {5000};
  pc.cuq = {0, 300};
  pc.maxp = 400;
  PrefillPlan Q;
  kvp::plan_prefill(pc.ctx.data(), pc.cuq.data(), 1, pc.maxp, pc.Hq, pc.Hkv, &Q);
  for (auto& it : Q.items)
    if (it.seq >= 0) {
      PrefillPlan b = Q;
      for (auto& jt : b.items)
        if (jt.seq >= 0) {
          jt.seq = -1;  // a tile never computed
          --b.real_items;
          break;
        }
      ++planted;
      if (!check_prefill(pc, b)) ++rejected;
      break;
    }
  {
    // one XCD given a workgroup past its share of the round
    PrefillPlan b = Q;
    size_t last = 0;
    for (size_t j = 0; j < b.items.size(); ++j)
      if (b.items[j].seq >= 0) last = j;
    const PrefillItem moved = b.items[last];
    b.items[last].seq = -1;
    b.items.resize((size_t)kvp::kPrefillSplitTarget + 8, PrefillItem{-1, 0, 0, 0, 0, -1, {0, 0}});
    b.items[(size_t)kvp::kPrefillSplitTarget + last % 8] = moved;
    ++planted;
    if (!check_prefill(pc, b)) ++rejected;
  }
  std::printf("self-test: %d of %d planted mistakes rejected\n", rejected, planted);
  return planted > 0 && rejected == planted;
}

int main(int argc, char** argv) {
  if (argc > 1 && !std::strcmp(argv[1], "self-test")) return self_test() ? 0 : 1;
  const int iters = argc > 1 ? std::atoi(argv[1]) : 200;
  rng.seed(argc > 2 ? std::strtoull(argv[2], nullptr, 10) : 12345);
  if (!run_errors()) return 1;
  for (int k = 0; k < iters; ++k) {
    if (!run_decode(random_decode())) {
      std::fprintf(stderr, "decode case %d\n", k);
      return 1;
    }
    if (!run_prefill(random_prefill())) {
      std::fprintf(stderr, "prefill case %d\n", k);
      return 1;
    }
  }
  std::printf("ok: %d decode and %d prefill plans checked (%d sessions with a split history)\n", iters, iters,
              g_split_sessions);
  return g_fail;
}
