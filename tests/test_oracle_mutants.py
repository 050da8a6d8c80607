"""Planted mistakes in the oracle are caught by its pins (CPU).

Each case plants one plausible mistake into the oracle (monkeypatched, on
the CPU, for the duration of the case) and runs the pin tests against it;
at least one pin must fail.  This is what backs the claim that the pins
would notice a dropped term, a wrong index or a wrong sign, rather than only
agreeing with the oracle as written.
"""

import numpy as np
import pytest

import oracle
import oracle.admission as adm
import oracle.fnv as ofnv
import oracle.keys as okeys
import oracle.layout as olayout
import oracle.restore as orest
import oracle.store as ostore
import oracle.tag as otag
import test_oracle_admission as t_adm
import test_oracle_failures as t_fail
import test_oracle_fnv_tag as t_fnv
import test_oracle_law as t_law
import test_oracle_probe as t_probe
import test_oracle_restore as t_rest
from oracle.fnv import fnv1a64


def _pins():
    """(name, callable) of the pin tests the mutants are run against."""
    law = t_law.LAW
    pins = [
        ("restore brute force, workload 1", t_rest.test_config1_bruteforce_and_counters),
        ("planar block layout", t_rest.test_planar_block_layout_config2_shape),
        ("identity table = concatenate", t_rest.test_identity_table_block_equals_chunk_is_concatenate),
        ("chain brute force", t_probe.test_chain_brute_force_tiny),
        ("chain prefix sensitivity", t_probe.test_chain_prefix_sensitivity),
        ("probe hole", t_probe.test_hole_gives_prefix_but_bitmap_shows_later_hits),
        ("workload 3 prefix", t_probe.test_config3_prefix_is_exactly_75_percent),
        ("engine-reported invalid group", t_fail.test_group_reported_invalid_without_window_failure),
        ("group fault collapses all groups", t_fail.test_group_fault_in_one_group_collapses_every_group),
        ("tag word loop", t_fnv.test_tag_matches_word_loop),
        ("admission exact fit", t_adm.test_exact_fit_and_release),
        ("admission lock", t_adm.test_budget_zero_is_a_lock),
        ("FNV-1a published vectors", lambda: [t_fnv.test_fnv1a64_published_vectors(e, d) for e, d in t_fnv._vectors()]),
        ("one group missing shortens the prefix", t_probe.test_one_group_missing_before_probe_shortens_prefix),
        ("abort after a window", t_fail.test_abort_after_window),
        ("slot offsets aligned", t_rest.test_slot_offsets_align_every_group_to_256),
    ]
    for s in range(3):
        pins.append((f"random layout brute force {s}", lambda s=s: t_rest.test_random_layout_bruteforce(s)))
    for W, mib in law["w_sweep_256k"]["rows"]:
        pins.append((f"window law W={W}", lambda W=W, mib=mib: t_law.test_window_law(W, mib)))
    pins.append(("bounded admission closed form",
                 lambda: t_adm.test_bounded_window_admits_floor_b_over_wc(8, 2)))
    return pins


def _caught(pins):
    """Names of the pins that fail (an assertion, or an error the mistake causes)."""
    failed = []
    for name, fn in pins:
        try:
            fn()
        except Exception:  # noqa: BLE001 -- any failure of a pin counts
            failed.append(name)
    return failed


# ---- the mistakes ------------------------------------------------------------
def _planar_plane_offset(mp):
    def place(layout, g, blk, o, recs):
        gr = layout.groups[g]
        m, r = recs.shape
        if gr.kind == "contig":
            blk[o * r:(o + m) * r] = recs.reshape(-1)
        else:
            s = gr.split_bytes
            blk[o * s:(o + m) * s] = recs[:, :s].reshape(-1)
            # the second plane placed without skipping the first one
            blk[o * (r - s):(o + m) * (r - s)] = recs[:, s:].reshape(-1)
    mp.setattr(orest, "_place", place)


def _block_index_ignores_table(mp):
    orig = orest.install_chunk

    def install(layout, i, slot, block_tables, pools):
        ident = [np.arange(len(bt)) for bt in block_tables]
        return orig(layout, i, slot, ident, pools)
    mp.setattr(orest, "install_chunk", install)


def _prefix_counts_every_hit(mp):
    orig = orest.probe

    def probe(store, tokens, chunk_tokens, salt, force_local=False):
        n, bm, keys = orig(store, tokens, chunk_tokens, salt, force_local)
        return int(bm.sum()), bm, keys
    mp.setattr(orest, "probe", probe)
    mp.setattr(oracle, "probe", probe)


def _chain_drops_previous_key(mp):
    def chain(tokens, chunk_tokens, salt):
        out = []
        for i in range(len(tokens) // chunk_tokens):
            d = okeys.chunk_digest(tokens[i * chunk_tokens:(i + 1) * chunk_tokens])
            out.append(fnv1a64(salt.to_bytes(8, "little") + d.to_bytes(8, "little")))
        return out
    for mod in (okeys, orest, oracle):
        mp.setattr(mod, "chain_keys", chain)


def _commit_drops_group_validity(mp):
    orig = orest.windowed_restore

    def restore(*a, **kw):
        kw.pop("invalid_groups", None)
        return orig(*a, **kw)
    mp.setattr(orest, "windowed_restore", restore)
    mp.setattr(oracle, "windowed_restore", restore)


def _window_never_released(mp):
    def trace(windows, slot_bytes):
        live, out = 0, [0]
        for win in windows:
            for _ in win:
                live += slot_bytes
                out.append(live)
            out.append(live)
        return out
    mp.setattr(orest, "live_trace", trace)


def _tag_sum_and_xor_swapped(mp):
    orig = otag.entry_tag

    def tag(data):
        t = orig(data)
        return ((t & 0xFFFFFFFF) << 32) | (t >> 32)
    for mod in (otag, ostore, orest, oracle, t_fnv):
        mp.setattr(mod, "entry_tag", tag)


def _admission_strict_budget(mp):
    def replay(budget, max_bound, W, slot_bytes, events):
        bound, tr = {}, adm.AdmissionTrace()
        for ev in events:
            if ev[0] == "end":
                bound.pop(ev[1], None)
                continue
            need = adm.plan_staging(W, ev[2], slot_bytes)
            if budget == 0:
                out = adm.OK if not bound else adm.BUSY
            elif need > budget:
                out = adm.TOO_LARGE
            elif sum(bound.values()) + need >= budget or len(bound) >= max_bound:   # >= instead of >
                out = adm.BUSY
            else:
                out = adm.OK
            if out == adm.OK:
                bound[ev[1]] = need
                tr.peak_bound_bytes = max(tr.peak_bound_bytes, sum(bound.values()))
                tr.peak_bound = max(tr.peak_bound, len(bound))
            elif out == adm.BUSY:
                tr.refused_busy += 1
            tr.outcomes.append(out)
        return tr
    mp.setattr(adm, "replay", replay)


def _admission_end_releases_nothing(mp):
    orig = adm.replay

    def replay(budget, max_bound, W, slot_bytes, events):
        return orig(budget, max_bound, W, slot_bytes, [e for e in events if e[0] != "end"])
    mp.setattr(adm, "replay", replay)


def _fnv1_instead_of_fnv1a(mp):
    def fnv1(data, h=ofnv.FNV64_OFFSET_BASIS):
        for octet in data:      # multiply before the XOR: FNV-1, not FNV-1a
            h = (h * ofnv.FNV64_PRIME) & ofnv.MASK64
            h ^= octet
        return h
    for mod in (ofnv, okeys, t_fnv):
        mp.setattr(mod, "fnv1a64", fnv1)


def _fnv_prime_off_by_two(mp):
    def f(data, h=ofnv.FNV64_OFFSET_BASIS):
        for octet in data:
            h ^= octet
            h = (h * (ofnv.FNV64_PRIME + 2)) & ofnv.MASK64
        return h
    for mod in (ofnv, okeys, t_fnv):
        mp.setattr(mod, "fnv1a64", f)


def _slot_groups_not_aligned(mp):
    mp.setattr(olayout, "align_up", lambda x, a=olayout.ALIGN: x)


def _commit_ignores_failed_window(mp):
    orig = orest.windowed_restore

    def restore(layout, store, keys, n_hit, W, block_tables, pools, valid, **kw):
        res = orig(layout, store, keys, n_hit, W, block_tables, pools, valid, **kw)
        if res.fail_reason != orest.FAIL_NONE and all(res.q):   # Q computed from q_g alone
            orest.set_request_valid(layout, n_hit, block_tables, valid, 1)
            res.exposed_tokens, res.fallback = n_hit * layout.chunk_tokens, 0
        return res
    mp.setattr(orest, "windowed_restore", restore)
    mp.setattr(oracle, "windowed_restore", restore)


def _invalidate_failed_groups_only(mp):
    orig = orest.windowed_restore

    def restore(layout, store, keys, n_hit, W, block_tables, pools, valid, **kw):
        res = orig(layout, store, keys, n_hit, W, block_tables, pools, valid, **kw)
        if res.fallback:        # groups that did not fail keep their blocks valid
            for g, gr in enumerate(layout.groups):
                if res.q[g]:
                    for k in range(orest.request_blocks(n_hit, layout.chunk_tokens, gr.block_tokens)):
                        valid[g][int(block_tables[g][k])] = 1
        return res
    mp.setattr(orest, "windowed_restore", restore)
    mp.setattr(oracle, "windowed_restore", restore)


def _probe_any_group(mp):
    def probe(store, tokens, chunk_tokens, salt, force_local=False):
        keys = okeys.chain_keys(tokens, chunk_tokens, salt)
        bitmap = np.zeros(len(keys), dtype=np.uint8)
        if force_local:
            return 0, bitmap, keys
        for i, h in enumerate(keys):     # any group's entry instead of every group's
            bitmap[i] = any(store.has(h, g) for g in range(store.n_groups))
        n = 0
        while n < len(keys) and bitmap[n]:
            n += 1
        return n, bitmap, keys
    mp.setattr(orest, "probe", probe)
    mp.setattr(oracle, "probe", probe)


def _install_mapping(mp, in_block_offset=True, tensor_major=True):
    def install(layout, i, slot, block_tables, pools):
        C = layout.chunk_tokens
        offs = layout.group_offsets()
        for g, gr in enumerate(layout.groups):
            flat = slot[offs[g]:offs[g] + layout.payload_bytes(g)]
            region = (flat.reshape(gr.n_tensors, C, gr.record_bytes) if tensor_major
                      else flat.reshape(C, gr.n_tensors, gr.record_bytes).transpose(1, 0, 2))
            for t in range(gr.n_tensors):
                q = 0
                while q < C:
                    k, o = divmod(i * C + q, gr.block_tokens)
                    m = min(gr.block_tokens - o, C - q)
                    orest._place(layout, g, pools[g][t, int(block_tables[g][k])],
                                 o if in_block_offset else 0, region[t, q:q + m])
                    q += m
    mp.setattr(orest, "install_chunk", install)


def _in_block_offset_dropped(mp):
    _install_mapping(mp, in_block_offset=False)


def _tensor_and_token_axes_swapped(mp):
    _install_mapping(mp, tensor_major=False)


MUTANTS = {
    "planar plane offset": _planar_plane_offset,
    "block index ignores the table": _block_index_ignores_table,
    "prefix counts every hit": _prefix_counts_every_hit,
    "chain drops the previous key": _chain_drops_previous_key,
    "commit drops a group's q_g": _commit_drops_group_validity,
    "window never released": _window_never_released,
    "tag sum and xor swapped": _tag_sum_and_xor_swapped,
    "admission budget strict": _admission_strict_budget,
    "admission end releases nothing": _admission_end_releases_nothing,
    "FNV-1 instead of FNV-1a": _fnv1_instead_of_fnv1a,
    "FNV prime off by two": _fnv_prime_off_by_two,
    "slot groups not 256-aligned": _slot_groups_not_aligned,
    "commit ignores a failed window": _commit_ignores_failed_window,
    "invalidate the failed groups only": _invalidate_failed_groups_only,
    "probe accepts any group": _probe_any_group,
    "in-block token offset dropped": _in_block_offset_dropped,
    "tensor and token axes swapped": _tensor_and_token_axes_swapped,
}


def test_unmutated_oracle_passes_every_pin():
    assert _caught(_pins()) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    MUTANTS[name](monkeypatch)
    failed = _caught(_pins())
    assert failed, f"no pin caught the planted mistake: {name}"
