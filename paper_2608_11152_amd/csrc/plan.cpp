// Host planner: validates host metadata and builds the work lists of the decode and prefill kernels.
// Deterministic: a plan depends only on lengths, group structure, head counts and the pool's element
// type, never on physical page ids, so GPU results are bitwise reproducible under any page permutation.
#include <algorithm>
#include <cmath>
#include <cstdio>
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

Status plan_decode(const int32_t* seq_lens, int B, int maxp, const kvp_group_prefix* gp, int Hq, int Hkv,
                   DecodePlan* plan, int chunk_start_pages) {
  *plan = DecodePlan();
  if (B < 0) return fail(KVP_EINVAL, "num_seqs %ld < 0", B);
  if (B > 0 && !seq_lens) return fail(KVP_EINVAL, "seq_lens is NULL");
  if (!supported_gqa(Hq, Hkv))
    return fail(KVP_EUNSUPPORTED, "num_q_heads %ld / num_kv_heads %ld: ratio must be 1, 2, 4, 8 or 16", Hq, Hkv);
  if (maxp < 0) return fail(KVP_EINVAL, "maxp %ld < 0", maxp);
  if (chunk_start_pages < 0) return fail(KVP_EINVAL, "chunk_start_pages %ld < 0", chunk_start_pages);
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

  // Members of each group that decode (seq_len > 0), in sequence order: group g's are
  // mem_list[mem_start[g] .. mem_start[g + 1]).
  const int NG = (gp ? gp->num_groups : 0);
  std::vector<int> mem_start(NG + 1, 0), mem_list;
  for (int i = 0; i < B; ++i)
    if (seq_lens[i] > 0 && shared_of(i) > 0) ++mem_start[gp->group_id[i] + 1];
  for (int g = 0; g < NG; ++g) mem_start[g + 1] += mem_start[g];
  mem_list.resize(mem_start[NG]);
  {
    std::vector<int> fill(mem_start.begin(), mem_start.end() - 1);
    for (int i = 0; i < B; ++i)
      if (seq_lens[i] > 0 && shared_of(i) > 0) mem_list[fill[gp->group_id[i]]++] = i;
  }
  auto n_mem = [&](int g) { return mem_start[g + 1] - mem_start[g]; };

  // Units: contiguous page ranges read for one set of query columns.  A group's shared prompt pages
  // form one unit per subgroup (at most 64 query columns, or 16 when wide groups go to the wave path,
  // see below), so the pages are read once per subgroup; each sequence's pages after its shared prefix
  // form one private unit.
  // A unit's members (the sequences owning its query columns) are plan->members[mem_off, +n_mem): a
  // group unit's are stored once and shared by all its chunks; a private unit's member is its row.
  struct Unit {
    int kind, row, lo, hi, tok_end, mem_off, n_mem;
  };
  std::vector<Unit> wave_units, group_units;
  wave_units.reserve(B + NG);
  std::vector<int> group_unit_of(B, -1), wave_unit_of(B, -1);  // shared-prefix unit of each member
  // Groups wider than one wave's 16 columns normally take the LDS-staged path, whose 4-wave blocks keep
  // the whole call on 4-wave workgroups.  When reading their prompt pages once per 16-column subgroup
  // instead adds at most 1% to the call's pages, they are planned as wave items: the call is then
  // wave-only and launches in 8-wave workgroups, which reach the CUs twice as fast.  Measured: the
  // mixed step (0.3% extra pages) 1% faster with bf16 pages and 4% with FP8 pages; the RLVR batch
  // (2.5% extra) 10% slower, so it stays on the LDS path.
  const int per_wave_sub = std::max(1, kMaxColsPerWave / G), per_group_sub = std::max(1, kMaxColsPerGroup / G);
  int64_t call_pages = 0, extra_pages = 0;
  for (int i = 0; i < B; ++i)
    if (seq_lens[i] > 0) call_pages += (seq_lens[i] + kPage - 1) / kPage - shared_of(i);
  for (int g = 0; g < NG; ++g) {
    const int64_t m = n_mem(g), S = gp->shared_pages[g];
    if (m == 0) continue;
    const int64_t n_group = (m + per_group_sub - 1) / per_group_sub, n_wave = (m + per_wave_sub - 1) / per_wave_sub;
    call_pages += n_group * S;
    if (m * G > kMaxColsPerWave) extra_pages += (n_wave - n_group) * S;
  }
  const bool wide_on_waves = extra_pages * 100 <= call_pages;
  const int per_sub = wide_on_waves ? per_wave_sub : per_group_sub;
  plan->members.reserve(mem_list.size() + B);
  for (int g = 0; g < NG; ++g) {
    const int S = gp->shared_pages[g];
    for (int m0 = mem_start[g]; m0 < mem_start[g + 1]; m0 += per_sub) {
      const int m1 = std::min(mem_start[g + 1], m0 + per_sub);
      Unit u{1, mem_list[m0], 0, S, S * kPage, (int)plan->members.size(), m1 - m0};
      plan->members.insert(plan->members.end(), mem_list.begin() + m0, mem_list.begin() + m1);
      const bool wide = u.n_mem * G > kMaxColsPerWave;
      for (int k = m0; k < m1; ++k)
        (wide ? group_unit_of : wave_unit_of)[mem_list[k]] = (int)(wide ? group_units : wave_units).size();
      (wide ? group_units : wave_units).push_back(u);
    }
  }
  for (int i = 0; i < B; ++i) {
    if (seq_lens[i] <= 0) continue;
    const int lo = shared_of(i);
    const int hi = (seq_lens[i] + kPage - 1) / kPage;
    if (hi > lo) {
      wave_units.push_back(Unit{0, i, lo, hi, seq_lens[i], (int)plan->members.size(), 1});
      plan->members.push_back(i);
    }
  }

  // Wave-path units are cut into equal segments of consecutive pages ("stream-K" over the concatenated
  // unit list): segment s is processed by waves s*Hkv .. s*Hkv+Hkv-1 (one per KV head), so every wave
  // streams the same number of pages whatever the length skew, and a sequence is split only where a
  // segment boundary falls inside it.  About kDecodeWaves waves: one round of the waves that
  // are resident at once on 256 CUs.  Segments hold at least 8 pages (128 tokens): a chunk's partial
  // (G x d fp32 written, then read by the merge) stays within ~6% of its KV bytes, and a call too small
  // for the budget (a few long sequences) still spreads over many waves instead of a few long ones.
  int64_t total_pages = 0, group_pages = 0;
  for (const Unit& u : wave_units) total_pages += u.hi - u.lo;
  for (const Unit& u : group_units) group_pages += u.hi - u.lo;
  // The LDS-staged shared-prefix blocks run in the same launch, after the wave blocks in grid order.
  // Reserve block slots for them out of the one-round budget (4 waves per block), in proportion to
  // their share of the pages weighted by their lower per-block throughput (about 2.5x less than four
  // independent streaming waves), so they drain while the wave segments run instead of after them.
  const int64_t budget_blocks = std::max<int64_t>(1, kDecodeWaves / 4);
  int64_t reserve = 0;
  if (group_pages > 0) {
    const double wg = 2.5 * (double)group_pages, ww = (double)total_pages;
    reserve = (int64_t)std::ceil((double)budget_blocks * wg / (wg + ww));
    reserve = std::max<int64_t>(1, std::min<int64_t>(reserve, budget_blocks / 2));
  }
  plan->group_reserved_blocks = (int)reserve;
  const int64_t segs_target = std::max<int64_t>(1, (budget_blocks - reserve) * 4 / Hkv);
  int64_t seg_pages = (total_pages + segs_target - 1) / segs_target;
  seg_pages = std::max<int64_t>(kMinSegmentPages, (seg_pages + 1) & ~int64_t(1));

  struct Chunk { int unit, lo, hi; };
  std::vector<Chunk> wave_chunks;
  std::vector<int> seg_of_chunk;
  wave_chunks.reserve(wave_units.size() + segs_target + 1);
  seg_of_chunk.reserve(wave_units.size() + segs_target + 1);
  std::vector<int> n_chunks_wave(wave_units.size(), 0);
  {
    // A chunk's start costs a wave about chunk_start_pages pages of streaming (its item, the query
    // fragments and the first page ids are dependent reads), so a segment's budget counts each chunk
    // as its pages plus that start: segments that span several units hold fewer pages.  The budget is
    // the smallest at which the cut still fits segs_target segments (one round of waves).
    const int64_t K = chunk_start_pages;
    auto cut = [&](int64_t cap, bool emit) -> int64_t {  // returns the segment count
      int64_t fill = 0;
      int seg = 0;
      for (size_t u = 0; u < wave_units.size(); ++u) {
        int lo = wave_units[u].lo;
        while (lo < wave_units[u].hi) {
          if (fill > 0 && fill + K >= cap) {  // no room for another start and a page
            fill = 0;
            ++seg;
          }
          fill += K;
          const int take = (int)std::min<int64_t>(wave_units[u].hi - lo, cap - fill);
          if (emit) {
            wave_chunks.push_back(Chunk{(int)u, lo, lo + take});
            seg_of_chunk.push_back(seg);
            n_chunks_wave[u]++;
          }
          lo += take;
          fill += take;
          if (fill >= cap) {
            fill = 0;
            ++seg;
          }
        }
      }
      return fill > 0 ? seg + 1 : seg;
    };
    int64_t cap = seg_pages + K;  // a single-chunk segment still holds seg_pages pages
    if (cut(cap, false) > segs_target) {
      int64_t lo = cap, hi = 2 * cap;
      while (cut(hi, false) > segs_target) hi *= 2;
      while (lo + 1 < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        (cut(mid, false) > segs_target ? lo : hi) = mid;
      }
      cap = hi;
    }
    cut(cap, true);
    plan->pages_per_split = (int)(cap - K);
  }
  // Wide shared-prefix units (LDS-staged workgroup kernel): fixed chunks of kGroupChunkPages pages.
  std::vector<Chunk> group_chunks;
  std::vector<int> n_chunks_group(group_units.size(), 0);
  for (size_t u = 0; u < group_units.size(); ++u)
    for (int lo = group_units[u].lo; lo < group_units[u].hi; lo += kGroupChunkPages) {
      group_chunks.push_back(Chunk{(int)u, lo, std::min(group_units[u].hi, lo + kGroupChunkPages)});
      n_chunks_group[u]++;
    }

  // Partial slots: per sequence, its shared-prefix chunks first (the same slot index for every member
  // of a subgroup), then its private chunks.  A sequence with a single private chunk and no prefix
  // writes its output directly (slot -1) and needs no merge.
  std::vector<int> n_prefix(B, 0), n_priv(B, 0);
  for (int i = 0; i < B; ++i) {
    if (group_unit_of[i] >= 0) n_prefix[i] = n_chunks_group[group_unit_of[i]];
    if (wave_unit_of[i] >= 0) n_prefix[i] = n_chunks_wave[wave_unit_of[i]];
  }
  for (size_t u = 0; u < wave_units.size(); ++u)
    if (wave_units[u].kind == 0) n_priv[wave_units[u].row] = n_chunks_wave[u];
  plan->part_base.assign(B, 0);
  plan->n_parts.assign(B, 0);
  int32_t total = 0;
  for (int i = 0; i < B; ++i) {
    const int np = n_prefix[i] + n_priv[i];
    const bool direct = (n_prefix[i] == 0 && n_priv[i] == 1);
    plan->n_parts[i] = direct ? 1 : np;
    plan->part_base[i] = total;
    if (!direct) {
      total += np;
      plan->merge_seqs.push_back(i);
    }
  }
  plan->total_parts = total;

  auto emit = [&](const Unit& un, const Chunk& c, int k) {
    DecodeItem it{un.kind, un.row, c.lo, c.hi, un.tok_end, un.mem_off, un.n_mem, 0};
    if (un.kind == 1) it.slot = k;
    else it.slot = (n_prefix[un.row] == 0 && n_priv[un.row] == 1) ? -1 : n_prefix[un.row] + k;
    return it;
  };
  {
    std::vector<int> k_of(wave_units.size(), 0);
    plan->seg_off.reserve(segs_target + 2);
    plan->wave_items.reserve(wave_chunks.size());
    plan->seg_off.push_back(0);
    for (size_t c = 0; c < wave_chunks.size(); ++c) {
      if (c > 0 && seg_of_chunk[c] != seg_of_chunk[c - 1]) plan->seg_off.push_back((int)c);
      const int u = wave_chunks[c].unit;
      plan->wave_items.push_back(emit(wave_units[u], wave_chunks[c], k_of[u]++));
    }
    plan->seg_off.push_back((int)wave_chunks.size());
    if (wave_chunks.empty()) plan->seg_off.assign(1, 0);
  }
  {
    std::vector<int> k_of(group_units.size(), 0);
    for (const Chunk& c : group_chunks) plan->group_items.push_back(emit(group_units[c.unit], c, k_of[c.unit]++));
  }
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
  // History split.  Long histories under few query tiles (a short uncached suffix over a long cached
  // prefix, Eq. 1) would leave most CUs idle: each tile streams its whole history alone.  When the
  // call's tiles are fewer than kPrefillSplitTarget, each tile's 64-key stages are cut into ranges of
  // about T stages.  T starts where the call would hold about kPrefillSplitTarget ranges (at least
  // kPrefillMinSplitStages stages each) and grows until the ranges fit the resident workgroups in one
  // round: a range past that would wait for a whole range to finish.  A range may start only at a stage
  // whose first key every query row of the session sees (st * 64 <= ctx), so every range is non-empty
  // for every row; the ranges of one session are shared by all its tiles and the last one runs to each
  // tile's own last stage.
  auto n_tiles = [&](int i) { return (int)(((int64_t)(cu_q[i + 1] - cu_q[i]) * G + kPrefillRows - 1) / kPrefillRows); };
  // 64-key stages of every tile (its last row's keys), computed once: tile t of session i at tile_off[i] + t
  std::vector<int64_t> tile_off(B + 1, 0);
  for (int i = 0; i < B; ++i) tile_off[i + 1] = tile_off[i] + n_tiles(i);
  std::vector<int> tile_st(tile_off[B]);
  for (int i = 0; i < B; ++i) {
    const int64_t C = cu_q[i + 1] - cu_q[i];
    for (int t = 0; t < n_tiles(i); ++t) {
      const int64_t last_row = std::min<int64_t>(C * G - 1, (int64_t)t * kPrefillRows + kPrefillRows - 1);
      tile_st[tile_off[i] + t] = (int)((ctx_lens[i] + last_row / G + 1 + 63) / 64);
    }
  }
  auto tile_stages = [&](int i, int t) { return tile_st[tile_off[i] + t]; };
  std::vector<std::vector<int>> bounds(B);  // split starts after 0, per session
  auto split_with = [&](int64_t T) {        // bounds for ranges of about T stages; returns the range count
    int64_t ranges = 0;
    for (int i = 0; i < B; ++i) {
      bounds[i].clear();
      const int C = cu_q[i + 1] - cu_q[i];
      if (C == 0) continue;
      const int nst = tile_stages(i, 0);             // the session's shortest tile
      const int max_start = ctx_lens[i] / 64;        // latest stage a range may start at
      const int64_t want = (nst + T - 1) / T;
      const int S = (int)std::min<int64_t>(want, (int64_t)max_start + 1);
      for (int k = 1; k < S; ++k) {
        const int b = std::min<int>(max_start, (int)((int64_t)k * nst / S));
        if (b > (bounds[i].empty() ? 0 : bounds[i].back())) bounds[i].push_back(b);
      }
      ranges += (int64_t)n_tiles(i) * Hkv * ((int64_t)bounds[i].size() + 1);
    }
    return ranges;
  };
  plan->nsplit.assign(B, 1);
  plan->part_base.assign(B, 0);
  {
    int64_t tiles_total = 0, work = 0, longest_tile = 0;
    for (int i = 0; i < B; ++i) {
      const int nt = n_tiles(i);
      tiles_total += (int64_t)nt * Hkv;
      for (int t = 0; t < nt; ++t) {
        work += (int64_t)tile_stages(i, t) * Hkv;
        longest_tile = std::max<int64_t>(longest_tile, tile_stages(i, t));
      }
    }
    if (tiles_total > 0 && tiles_total < kPrefillSplitTarget) {
      int64_t lo = std::max<int64_t>(kPrefillMinSplitStages, (work + kPrefillSplitTarget - 1) / kPrefillSplitTarget);
      // The range count does not grow with T and is tiles_total (< the target) once T covers every
      // tile: the smallest T in [lo, longest_tile] that fits, by bisection.
      if (split_with(lo) > kPrefillSplitTarget) {
        int64_t hi = std::max(lo, longest_tile);
        while (lo + 1 < hi) {
          const int64_t mid = lo + (hi - lo) / 2;
          (split_with(mid) > kPrefillSplitTarget ? lo : hi) = mid;
        }
        split_with(hi);
      }
      for (int i = 0; i < B; ++i) plan->nsplit[i] = (int)bounds[i].size() + 1;
    }
  }
  int32_t parts = 0;
  for (int i = 0; i < B; ++i) {
    if (plan->nsplit[i] == 1) continue;
    const int C = cu_q[i + 1] - cu_q[i];
    plan->part_base[i] = parts;
    for (int j = 0; j < C; ++j) {
      const int32_t rec[4] = {cu_q[i] + j, parts + j * plan->nsplit[i], plan->nsplit[i], 0};
      plan->merge_info.insert(plan->merge_info.end(), rec, rec + 4);
    }
    if ((int64_t)parts + (int64_t)C * plan->nsplit[i] > INT32_MAX) return fail(KVP_EINVAL, "too many partials");
    parts += C * plan->nsplit[i];
  }
  plan->total_parts = parts;

  // Units = contiguous runs of query tiles of one (session, kv head, key range).  Tiles of a unit read
  // the same KV, so a unit is kept on one XCD (workgroup b runs on XCD b % 8) to share that XCD's L2.
  // Units are spread over the 8 XCDs longest-first; within an XCD the heaviest units start first.  When
  // the whole call fits the resident workgroups (one round), no XCD may take more than its share of
  // them: a unit that fits no XCD whole is dealt out tile by tile.
  struct Unit { int seq, kvh, t0, t1, k; double w; };
  std::vector<Unit> units;
  int64_t tiles_total = 0;
  for (int i = 0; i < B; ++i) tiles_total += (int64_t)n_tiles(i) * Hkv * plan->nsplit[i];
  const int64_t seg = std::max<int64_t>(1, tiles_total / 64);  // at least ~64 units to balance 8 XCDs
  auto range_of = [&](int i, int k, int t, int* lo, int* hi) {
    *lo = k == 0 ? 0 : bounds[i][k - 1];
    *hi = k + 1 < plan->nsplit[i] ? bounds[i][k] : tile_stages(i, t);
  };
  for (int i = 0; i < B; ++i) {
    const int nt = n_tiles(i);
    for (int h = 0; h < Hkv; ++h)
      for (int k = 0; k < plan->nsplit[i]; ++k)
        for (int t0 = 0; t0 < nt; t0 += (int)seg) {
          const int t1 = std::min<int>(nt, t0 + (int)seg);
          double w = 0;
          for (int t = t0; t < t1; ++t) {
            int lo, hi;
            range_of(i, k, t, &lo, &hi);
            w += hi - lo;
          }
          units.push_back(Unit{i, h, t0, t1, k, w});
        }
  }
  std::vector<int> order(units.size());
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return units[a].w > units[b].w; });
  constexpr int kXcd = 8;
  const bool one_round = tiles_total <= kPrefillSplitTarget;
  const size_t cap = one_round ? (size_t)(kPrefillSplitTarget / kXcd) : SIZE_MAX;
  std::vector<std::vector<PrefillItem>> bins(kXcd);
  for (auto& b : bins) b.reserve((size_t)(tiles_total / kXcd + seg + 1));
  std::vector<double> load(kXcd, 0.0);
  auto place = [&](int x, const Unit& un, int t) {
    int lo, hi;
    range_of(un.seq, un.k, t, &lo, &hi);
    load[x] += hi - lo;
    bins[x].push_back(PrefillItem{un.seq, un.kvh, t * kPrefillRows, lo, hi,
                                  plan->nsplit[un.seq] == 1 ? -1 : un.k, {0, 0}});
  };
  // the least-loaded XCD with room for n more workgroups, or -1
  auto pick = [&](size_t n) {
    int best = -1;
    for (int x = 0; x < kXcd; ++x)
      if (bins[x].size() + n <= cap && (best < 0 || load[x] < load[best])) best = x;
    return best;
  };
  for (int u : order) {
    const Unit& un = units[u];
    const int x = pick((size_t)(un.t1 - un.t0));
    if (x >= 0) {
      for (int t = un.t0; t < un.t1; ++t) place(x, un, t);
    } else {
      for (int t = un.t0; t < un.t1; ++t) {
        const int y = pick(1);  // total <= kXcd * cap: some XCD has room for one
        place(y >= 0 ? y : (int)(std::min_element(load.begin(), load.end()) - load.begin()), un, t);
      }
    }
  }
  size_t longest = 0;
  for (auto& b : bins) longest = std::max(longest, b.size());
  plan->items.assign(longest * kXcd, PrefillItem{-1, 0, 0, 0, 0, -1, {0, 0}});
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
