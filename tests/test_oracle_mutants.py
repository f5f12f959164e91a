"""Plant plausible mistakes in a copy of the oracle and check that the pins
in test_oracle.py catch every one of them (each mutant must fail a pin)."""
import os
import subprocess
import sys

import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.cpp")

MUTANTS = {
    "walk_continues_after_partial_edge": ("    d += k;\n    if (k < e) break;", "    d += k;"),
    "walk_counts_whole_edge": ("    d += k;\n    if (k < e) break;", "    d += e;\n    if (k < e) break;"),
    "hit_rounds_up": ("block_size * (w.matched / block_size)",
                      "block_size * ((w.matched + block_size - 1) / block_size)"),
    "demand_skips_root": ("c != nullptr; c = c->parent", "c->parent != nullptr; c = c->parent"),
    "split_forgets_counts": ("mid->pending_count = child->pending_count;", "mid->pending_count = 0;"),
    "cluster_accepts_count_one": ("if (node->pending_count >= 2) deepest = node;",
                                  "if (node->pending_count >= 1) deepest = node;"),
    "threshold_strict": ("share >= threshold", "share > threshold"),
    "id_is_largest_member": ("if (cluster[r] && !smallest_member.count(cluster[r])) smallest_member[cluster[r]] = r;",
                             "if (cluster[r]) smallest_member[cluster[r]] = r;"),
    "children_in_descending_order": ("for (auto it = n->kids.rbegin(); it != n->kids.rend(); ++it)",
                                     "for (auto it = n->kids.begin(); it != n->kids.end(); ++it)"),
    "split_depth_off_by_one": ("      mid->depth = node->depth + k;\n      child->edge.erase",
                               "      mid->depth = node->depth + k + 1;\n      child->edge.erase"),
    "reachability_check_dropped": ("if (seen != num_nodes) { free_tree(t); return nullptr; }", ""),
    "last_node_is_parent_on_partial": ("  return {d, c};", "  return {d, (c->parent && d < c->depth) ? c->parent : c};"),
    "evict_score_skips_self": ("for (const Node* a = t->by_canon[c]; a != nullptr; a = a->parent) {",
                               "for (const Node* a = t->by_canon[c]->parent; a != nullptr; a = a->parent) {"),
    "evict_largest_first": ("    const auto it = leaves.begin();", "    const auto it = std::prev(leaves.end());"),
    "evict_frees_inner_nodes_early": ("--kids_left[p->canon] == 0", "--kids_left[p->canon] <= 1"),
    "block_hit_counts_partial_block": ("for (int64_t b = 0; (b + 1) * B <= len; ++b) {",
                                       "for (int64_t b = 0; b * B < len; ++b) {"),
    "block_hash_not_chained": ("{ return k + digest; }", "{ return 0x243F6A8885A308D3ULL + digest + 0 * k; }"),
    "block_digest_ignores_its_index": (" ^ (0x9E3779B97F4A7C15ULL * (uint64_t)(idx + 1)));", ");"),
    "nh_without_position_keys": ("const uint32_t x = (uint32_t)blk[i] + nh_key(i, pass);",
                                 "const uint32_t x = (uint32_t)blk[i];"),
    "nh_single_pass": ("for (int pass = 0; pass < 2; ++pass)", "for (int pass = 0; pass < 1; ++pass)"),
    "block_hashes_never_stored": ("        stored.insert(st.k);\n", ""),
    "offline_count_ascending": ("if (a->count != b->count) return a->count > b->count;",
                                "if (a->count != b->count) return a->count < b->count;"),
    "offline_ties_by_latest": ("    return a->first < b->first;\n  });", "    return a->first > b->first;\n  });"),
    "offline_ends_reversed": ("for (int64_t r : v->ends) out[(*k)++] = r;",
                              "for (auto it = v->ends.rbegin(); it != v->ends.rend(); ++it) out[(*k)++] = *it;"),
    "offline_ignores_depth_limit": ("const int64_t t = len < depth_limit ? len : depth_limit;", "const int64_t t = len;"),
    "score_leaves_out_own_request": ("      score += node->pending_count * node->elen;",
                                     "      score += (node->pending_count - 1) * node->elen;"),
    "score_weights_by_depth": ("      score += node->pending_count * node->elen;",
                               "      score += node->pending_count * node->depth;"),
    "warm_is_at_least_tau": ("section_out[r] = h[r] > tau ? 0", "section_out[r] = h[r] >= tau ? 0"),
    "pioneer_is_the_latest": ("it->second = std::min(it->second, r);", "it->second = std::max(it->second, r);"),
    "section_prefix_too_short": ("const int64_t k = len < theta ? len : theta;",
                                 "const int64_t k = len < theta - 1 ? len : theta - 1;"),
    "sharing_counts_single_requests": ("if (kv.second->pending_count >= 2) sharing = 1;",
                                       "if (kv.second->pending_count >= 1) sharing = 1;"),
}

PINS = "brute_force or worked or unary or invalid or tiny or agentic or hashed or mix64 or offline"


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    mutant = tmp_path / "oracle_mutant.cpp"
    mutant.write_text(src.replace(old, new))
    lib = O.build(force=True, src=str(mutant), out=str(tmp_path / "liboracle_mutant.so"))
    env = dict(os.environ, PEEK_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle.py"), "-k", PINS],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
