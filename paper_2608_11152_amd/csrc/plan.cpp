// Host planner: validates host metadata and builds the work lists of the decode and prefill kernels.
// Deterministic: a plan depends only on lengths, group structure and head counts, never on physical
// page ids, so GPU results are bitwise reproducible under any page permutation.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <numeric>

#include "kvp_plan.h"

namespace kvp {

static Status fail(int code, const char* fmt, long a = 0, long b = 0, long c = 0) {
  Status s;
  s.code = code;
  char buf[256];
  std::snprintf(buf, sizeof(buf), fmt, a, b, c);
  s.msg = buf;
  return s;
}

static bool supported_gqa(int Hq, int Hkv) {
  if (Hq <= 0 || Hkv <= 0 || Hq % Hkv) return false;
  const int G = Hq / Hkv;
  return G == 1 || G == 2 || G == 4 || G == 8 || G == 16;
}

Status validate_group_prefix(const int32_t* lens, int B, const kvp_group_prefix* gp) {
  if (!gp) return {};
  if (gp->num_groups < 0) return fail(KVP_EINVAL, "num_groups %ld < 0", gp->num_groups);
  if (gp->num_groups > 0 && (!gp->group_id || !gp->shared_pages))
    return fail(KVP_EINVAL, "group_prefix arrays are NULL");
  if (gp->num_groups == 0) return {};
  if (!gp->group_id) return fail(KVP_EINVAL, "group_id is NULL");
  for (int g = 0; g < gp->num_groups; ++g)
    if (gp->shared_pages[g] < 0) return fail(KVP_EGROUP, "shared_pages[%ld] = %ld < 0", g, gp->shared_pages[g]);
  for (int i = 0; i < B; ++i) {
    const int g = gp->group_id[i];
    if (g < -1 || g >= gp->num_groups) return fail(KVP_EGROUP, "group_id[%ld] = %ld out of range", i, g);
    if (g >= 0 && lens && lens[i] > 0 && (int64_t)gp->shared_pages[g] * kPage > lens[i])
      return fail(KVP_EGROUP, "sequence %ld (len %ld) is shorter than its group's shared prefix (%ld pages)",
                  i, lens[i], gp->shared_pages[g]);
  }
  return {};
}

// Target number of decode waves per call.  KVP_DECODE_WAVES overrides the default for tuning sweeps;
// the plan stays a pure function of its inputs for a given value.
static int64_t decode_target_waves() {
  static const int64_t v = [] {
    const char* e = std::getenv("KVP_DECODE_WAVES");
    const long x = e ? std::strtol(e, nullptr, 10) : 0;
    return x > 0 ? (int64_t)x : (int64_t)4096;
  }();
  return v;
}

// Split [lo, hi) pages into nearly equal ranges of at most `ch` pages; interior boundaries are even so
// that the kernels' two-page steps never straddle a boundary.
static void split_range(int lo, int hi, int ch, std::vector<std::pair<int, int>>* out) {
  out->clear();
  const int n = hi - lo;
  if (n <= 0) return;
  const int parts = (n + ch - 1) / ch;
  int len = (n + parts - 1) / parts;
  len = (len + 1) & ~1;
  for (int a = lo; a < hi; a += len) out->emplace_back(a, std::min(hi, a + len));
}

Status plan_decode(const int32_t* seq_lens, int B, int maxp, const kvp_group_prefix* gp, int Hq, int Hkv,
                   DecodePlan* plan) {
  *plan = DecodePlan();
  if (B < 0) return fail(KVP_EINVAL, "num_seqs %ld < 0", B);
  if (B > 0 && !seq_lens) return fail(KVP_EINVAL, "seq_lens is NULL");
  if (!supported_gqa(Hq, Hkv))
    return fail(KVP_EUNSUPPORTED, "num_q_heads %ld / num_kv_heads %ld: ratio must be 1, 2, 4, 8 or 16", Hq, Hkv);
  if (maxp < 0) return fail(KVP_EINVAL, "maxp %ld < 0", maxp);
  for (int i = 0; i < B; ++i) {
    if (seq_lens[i] < 0) return fail(KVP_EINVAL, "seq_lens[%ld] = %ld < 0", i, seq_lens[i]);
    if ((int64_t)seq_lens[i] > (int64_t)maxp * kPage)
      return fail(KVP_ERANGE, "seq_lens[%ld] = %ld exceeds maxp * 16 = %ld", i, seq_lens[i], (long)maxp * kPage);
  }
  Status st = validate_group_prefix(seq_lens, B, gp);
  if (!st.ok()) return st;
  if (gp && gp->num_groups > 0)
    for (int g = 0; g < gp->num_groups; ++g)
      if (gp->shared_pages[g] > maxp) return fail(KVP_EGROUP, "shared_pages[%ld] = %ld > maxp", g, gp->shared_pages[g]);

  const int G = Hq / Hkv;
  auto shared_of = [&](int i) -> int {
    if (!gp || gp->num_groups == 0) return 0;
    const int g = gp->group_id[i];
    return g >= 0 ? gp->shared_pages[g] : 0;
  };

  // Members of each group that decode (seq_len > 0), in sequence order.
  const int NG = (gp ? gp->num_groups : 0);
  std::vector<std::vector<int>> mem(NG);
  for (int i = 0; i < B; ++i)
    if (seq_lens[i] > 0 && shared_of(i) > 0) mem[gp->group_id[i]].push_back(i);

  // Pages per split: aim for about decode_target_waves() waves (several rounds of the ~12 waves per CU
  // that fit on 256 CUs) so equal-sized splits balance across the chip; never below 32 pages (512 tokens),
  // so a split's partial (G x d fp32 written, then read by the merge) stays within ~2% of its KV bytes.
  int64_t page_heads = 0;
  for (int i = 0; i < B; ++i) {
    const int np = (seq_lens[i] + kPage - 1) / kPage;
    page_heads += (int64_t)(np - (seq_lens[i] > 0 ? shared_of(i) : 0)) * Hkv;
  }
  for (int g = 0; g < NG; ++g)
    if (!mem[g].empty()) page_heads += (int64_t)gp->shared_pages[g] * Hkv;
  const int64_t waves = decode_target_waves();
  int64_t ch = (page_heads + waves - 1) / waves;
  ch = std::max<int64_t>(32, std::min<int64_t>(1024, ch));
  ch = (ch + 1) & ~1;
  plan->pages_per_split = (int)ch;

  std::vector<int> n_prefix(B, 0), n_priv(B, 0);
  std::vector<std::pair<int, int>> rng;
  // Shared-prefix items: one per (subgroup, split).  A subgroup holds at most 64 query columns.
  struct Pending { DecodeItem it; std::vector<int> mems; };
  std::vector<Pending> prefix_items;
  for (int g = 0; g < NG; ++g) {
    if (mem[g].empty()) continue;
    const int S = gp->shared_pages[g];
    split_range(0, S, (int)ch, &rng);
    const int per_sub = std::max(1, kMaxColsPerGroup / G);
    for (size_t m0 = 0; m0 < mem[g].size(); m0 += per_sub) {
      const size_t m1 = std::min(mem[g].size(), m0 + per_sub);
      for (size_t k = 0; k < rng.size(); ++k) {
        Pending p;
        p.it = DecodeItem{1, mem[g][m0], rng[k].first, rng[k].second, S * kPage, 0, (int)(m1 - m0), (int)k};
        p.mems.assign(mem[g].begin() + m0, mem[g].begin() + m1);
        prefix_items.push_back(std::move(p));
      }
    }
    for (int i : mem[g]) n_prefix[i] = (int)rng.size();
  }
  // Private items: the pages after the shared prefix, split.
  std::vector<DecodeItem> priv;
  for (int i = 0; i < B; ++i) {
    if (seq_lens[i] <= 0) continue;
    const int lo = shared_of(i);
    const int hi = (seq_lens[i] + kPage - 1) / kPage;
    split_range(lo, hi, (int)ch, &rng);
    n_priv[i] = (int)rng.size();
    for (size_t k = 0; k < rng.size(); ++k)
      priv.push_back(DecodeItem{0, i, rng[k].first, rng[k].second, seq_lens[i], i, 1, n_prefix[i] + (int)k});
  }

  // Partial slots per sequence; a sequence with exactly one private split writes its output directly.
  plan->part_base.assign(B, 0);
  plan->n_parts.assign(B, 0);
  int32_t total = 0;
  for (int i = 0; i < B; ++i) {
    const int np = n_prefix[i] + n_priv[i];
    const bool direct = (np == 1 && n_priv[i] == 1);
    plan->n_parts[i] = direct ? 1 : np;
    plan->part_base[i] = total;
    if (!direct) total += np;
    if (!direct) plan->merge_seqs.push_back(i);
  }
  plan->total_parts = total;

  for (auto& p : prefix_items) {
    p.it.mem_off = (int)plan->members.size();
    plan->members.insert(plan->members.end(), p.mems.begin(), p.mems.end());
    if (p.it.n_mem * G <= kMaxColsPerWave) plan->wave_items.push_back(p.it);
    else plan->group_items.push_back(p.it);
  }
  for (auto it : priv) {
    it.mem_off = (int)plan->members.size();
    plan->members.push_back(it.row);
    if (n_prefix[it.row] + n_priv[it.row] == 1) it.slot = -1;
    plan->wave_items.push_back(it);
  }
  // Longest ranges first (stable, so the order stays a pure function of the inputs).
  auto longer = [](const DecodeItem& a, const DecodeItem& b) {
    return (a.page_hi - a.page_lo) > (b.page_hi - b.page_lo);
  };
  std::stable_sort(plan->wave_items.begin(), plan->wave_items.end(), longer);
  std::stable_sort(plan->group_items.begin(), plan->group_items.end(), longer);
  return {};
}

Status plan_prefill(const int32_t* ctx_lens, const int32_t* cu_q, int B, int maxp, int Hq, int Hkv,
                    PrefillPlan* plan) {
  *plan = PrefillPlan();
  if (B < 0) return fail(KVP_EINVAL, "num_seqs %ld < 0", B);
  if (B > 0 && (!ctx_lens || !cu_q)) return fail(KVP_EINVAL, "ctx_lens or cu_q is NULL");
  if (!supported_gqa(Hq, Hkv))
    return fail(KVP_EUNSUPPORTED, "num_q_heads %ld / num_kv_heads %ld: ratio must be 1, 2, 4, 8 or 16", Hq, Hkv);
  if (B > 0 && cu_q[0] != 0) return fail(KVP_EINVAL, "cu_q[0] = %ld, must be 0", cu_q[0]);
  const int G = Hq / Hkv;
  for (int i = 0; i < B; ++i) {
    const int C = cu_q[i + 1] - cu_q[i];
    if (C < 0) return fail(KVP_EINVAL, "cu_q decreases at %ld", i);
    if (ctx_lens[i] < 0) return fail(KVP_EINVAL, "ctx_lens[%ld] = %ld < 0", i, ctx_lens[i]);
    if ((int64_t)ctx_lens[i] + C > (int64_t)maxp * kPage)
      return fail(KVP_ERANGE, "ctx_lens[%ld] + chunk = %ld exceeds maxp * 16 = %ld", i,
                  (long)ctx_lens[i] + C, (long)maxp * kPage);
  }
  // Units = contiguous runs of query tiles of one (session, kv head).  Tiles of a unit read the same
  // KV, so a unit is kept on one XCD (workgroup b runs on XCD b % 8) to share that XCD's L2.  Units are
  // spread over the 8 XCDs longest-first; within an XCD the heaviest units start first.
  struct Unit { int seq, kvh, t0, t1; double w; };
  std::vector<Unit> units;
  int64_t tiles_total = 0;
  for (int i = 0; i < B; ++i) tiles_total += (int64_t)((cu_q[i + 1] - cu_q[i]) * G + kPrefillRows - 1) / kPrefillRows * Hkv;
  const int64_t seg = std::max<int64_t>(1, tiles_total / 64);  // at least ~64 units to balance 8 XCDs
  for (int i = 0; i < B; ++i) {
    const int C = cu_q[i + 1] - cu_q[i];
    const int nt = (C * G + kPrefillRows - 1) / kPrefillRows;
    for (int h = 0; h < Hkv; ++h)
      for (int t0 = 0; t0 < nt; t0 += (int)seg) {
        const int t1 = std::min<int>(nt, t0 + (int)seg);
        double w = 0;
        for (int t = t0; t < t1; ++t) w += ctx_lens[i] + std::min(C - 1, (t * kPrefillRows + kPrefillRows - 1) / G) + 1;
        units.push_back(Unit{i, h, t0, t1, w});
      }
  }
  std::vector<int> order(units.size());
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return units[a].w > units[b].w; });
  constexpr int kXcd = 8;
  std::vector<std::vector<PrefillItem>> bins(kXcd);
  std::vector<double> load(kXcd, 0.0);
  for (int u : order) {
    const int x = (int)(std::min_element(load.begin(), load.end()) - load.begin());
    load[x] += units[u].w;
    for (int t = units[u].t0; t < units[u].t1; ++t)
      bins[x].push_back(PrefillItem{units[u].seq, units[u].kvh, t * kPrefillRows, 0});
  }
  size_t longest = 0;
  for (auto& b : bins) longest = std::max(longest, b.size());
  plan->items.assign(longest * kXcd, PrefillItem{-1, 0, 0, 0});
  for (int x = 0; x < kXcd; ++x)
    for (size_t j = 0; j < bins[x].size(); ++j) plan->items[j * kXcd + x] = bins[x][j];
  plan->real_items = tiles_total;
  return {};
}

Status check_tables(const int32_t* bt, int maxp, const int32_t* lens, int B, int num_pages,
                    const kvp_group_prefix* gp) {
  if (B > 0 && (!bt || !lens)) return fail(KVP_EINVAL, "NULL block table or lengths");
  for (int i = 0; i < B; ++i) {
    if (lens[i] < 0 || (int64_t)lens[i] > (int64_t)maxp * kPage)
      return fail(KVP_ERANGE, "lens[%ld] = %ld outside [0, maxp*16]", i, lens[i]);
    const int np = (lens[i] + kPage - 1) / kPage;
    for (int p = 0; p < np; ++p) {
      const int id = bt[(int64_t)i * maxp + p];
      if (id < 0 || id >= num_pages)
        return fail(KVP_ERANGE, "block_tables[%ld][%ld] = %ld outside the pool", i, p, id);
    }
  }
  Status st = validate_group_prefix(lens, B, gp);
  if (!st.ok() || !gp || gp->num_groups == 0) return st;
  std::vector<int> first(gp->num_groups, -1);
  for (int i = 0; i < B; ++i) {
    const int g = gp->group_id[i];
    if (g < 0) continue;
    if (first[g] < 0) { first[g] = i; continue; }
    const int S = std::min(gp->shared_pages[g], maxp);
    for (int p = 0; p < S; ++p)
      if (bt[(int64_t)i * maxp + p] != bt[(int64_t)first[g] * maxp + p])
        return fail(KVP_EGROUP, "sequence %ld: shared page %ld differs from its group's first member %ld", i, p,
                    first[g]);
  }
  return {};
}

}  // namespace kvp
