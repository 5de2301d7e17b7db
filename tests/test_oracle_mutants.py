"""The pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a copy of ``oracle/tempokv_oracle.c`` (a
wrong shift or constant, a dropped term, a swapped or off-by-one index, a
boundary moved by one, a rule inverted), compiles it, and runs the pin tests
of the function it touches against it in a child process.  The case passes
only if some pin fails.  The frozen golden hash vectors are left out of those
runs: they were written by the oracle itself and only guard against
regressions, so they must not be what catches a mistake.

The composition of the hash (the position word, the chain constant, reading
ids as unsigned words) is this library's own definition, since the paper
defines none; the independent reference implementation in tests/ref_hash.py,
written from that documented definition, is the pin that catches a change to
any of them."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "tempokv_oracle.c")

HASH = ["tests/test_oracle_hash.py", "tests/test_oracle_hash_ref.py", "tests/test_oracle_properties.py"]
LOOKUP = ["tests/test_oracle_lookup.py"]
COPY = ["tests/test_oracle_copy.py", "tests/test_oracle_properties.py"]
COMMIT = ["tests/test_oracle_commit.py", "tests/test_oracle_properties.py"]
VALIDATE = ["tests/test_oracle_validate.py"]

# (name, pin tests, text in the oracle, planted replacement)
MUTANTS = [
    ("mix_shift_30", HASH, "z = (z ^ (z >> 30))", "z = (z ^ (z >> 29))"),
    ("mix_multiplier", HASH, "0xBF58476D1CE4E5B9ull", "0xBF58476D1CE4E5BBull"),
    ("mix_final_shift", HASH, "return z ^ (z >> 31);", "return z ^ (z >> 32);"),
    ("digest_xor_not_sum", HASH, "d += or_mix64(word);", "d ^= or_mix64(word);"),
    ("digest_drops_position", HASH, "+ ((uint64_t)(j + 1) << 32)", "+ ((uint64_t)1 << 32)"),
    ("chain_not_chained", HASH, "h = or_mix64(h ^ d ^ OR_GAMMA);", "h = or_mix64(seed ^ d ^ OR_GAMMA);"),
    ("chain_seed_ignored", HASH, "uint64_t h = seed;", "uint64_t h = 0;"),
    ("chain_block_off_by_one", HASH, "tokens + tok_off[r] + b * OR_HASH_BLOCK", "tokens + tok_off[r] + b * OR_HASH_BLOCK + 1"),
    ("position_word_offset", HASH, "((uint64_t)(j + 1) << 32)", "((uint64_t)(j + 2) << 32)"),
    ("position_word_unshifted_index", HASH, "((uint64_t)(j + 1) << 32)", "((uint64_t)j << 32)"),
    ("chain_constant_dropped", HASH, "h = or_mix64(h ^ d ^ OR_GAMMA);", "h = or_mix64(h ^ d);"),
    ("signed_token_words", HASH, "(uint64_t)(uint32_t)tok16[j]", "(uint64_t)(int64_t)tok16[j]"),
    ("lookup_not_prefix", LOOKUP, "if (s < 0) still_prefix = 0;", ""),
    ("lookup_first_block_key", LOOKUP, "uint64_t key = block_hash[blk_off[r] + (j + 1) * blocks_per_chunk - 1];\n"
     "            int32_t s = or_index_find", "uint64_t key = block_hash[blk_off[r] + j * blocks_per_chunk];\n"
     "            int32_t s = or_index_find"),
    ("jobs_retrieve_one_too_many", LOOKUP, "if (j < hit_chunks[r]) {", "if (j <= hit_chunks[r]) {"),
    ("jobs_store_indexed_chunks", LOOKUP, "if (s >= 0) continue;", "if (s >= 0 && 0) continue;"),
    ("jobs_no_dedup", LOOKUP, "if (seen) continue;", "if (seen && 0) continue;"),
    ("jobs_slots_reversed", LOOKUP, "store[ns].slot = free_slots[ns];", "store[ns].slot = free_slots[num_free - 1 - ns];"),
    ("jobs_dropped_not_counted", LOOKUP, "if (ns >= num_free) { nd++; continue; }", "if (ns >= num_free) { continue; }"),
    ("scatter_layer_plane_swapped", COPY, "int64_t src = jb->slot * slot_bytes\n"
     "                                    + ((((int64_t)l * 2 + kv)", "int64_t src = jb->slot * slot_bytes\n"
     "                                    + ((((int64_t)kv * lo->L + l)"),
    ("scatter_token_dropped", COPY, "int64_t dst = kv * lo->kv_stride + blk * lo->block_stride\n"
     "                                    + ((int64_t)t * HD + x)", "int64_t dst = kv * lo->kv_stride + blk * lo->block_stride\n"
     "                                    + ((int64_t)0 * HD + x)"),
    ("scatter_block_bound", COPY, "if (blk < 0 || blk >= lo->num_blocks) continue;\n                    for (int32_t t = 0; t < lo->B; t++)\n"
     "                        for (int64_t x = 0; x < HD; x++)\n                            for (int32_t c = 0; c < lo->e; c++) {\n"
     "                                int64_t src = jb->slot", "if (blk < 0 || blk > lo->num_blocks) continue;\n                    for (int32_t t = 0; t < lo->B; t++)\n"
     "                        for (int64_t x = 0; x < HD; x++)\n                            for (int32_t c = 0; c < lo->e; c++) {\n"
     "                                int64_t src = jb->slot"),
    ("job_chunk_bound", COPY, "((int64_t)jb->chunk + 1) * nseg > bt_stride", "(int64_t)jb->chunk * nseg > bt_stride"),
    ("gather_kv_stride_dropped", COPY, "\n                                int64_t src = kv * lo->kv_stride + blk * lo->block_stride",
     "\n                                int64_t src = blk * lo->block_stride"),
    ("layer_scatter_plane_dropped", COPY, "int64_t src = jb->slot * part_bytes\n                                + (((int64_t)kv * lo->C",
     "int64_t src = jb->slot * part_bytes\n                                + (((int64_t)0 * lo->C"),
    ("layer_gather_block_stride_dropped", COPY, "\n                            int64_t src = kv * lo->kv_stride + blk * lo->block_stride",
     "\n                            int64_t src = kv * lo->kv_stride + (blk / 2) * lo->block_stride"),

    ("gather_segment_off_by_one", COPY, "+ ((((int64_t)l * 2 + kv) * lo->C + (int64_t)i * lo->B + t) * HD + x) * lo->e + c;\n"
     "                                int64_t src", "+ ((((int64_t)l * 2 + kv) * lo->C + (int64_t)(i + 1) % nseg * lo->B + t) * HD + x) * lo->e + c;\n"
     "                                int64_t src"),
    ("scatter_source_segment", COPY, "(((int64_t)layer * 2 + kv) * lo->C + (int64_t)i * lo->B) * HD * lo->e",
     "(((int64_t)layer * 2 + kv) * lo->C + (int64_t)i) * HD * lo->e"),
    ("gather_source_first_not_last", COPY, "*blk_out = blk;\n        found = 1;", "if (!found) *blk_out = blk;\n        found = 1;"),
    ("commit_strict_laxity", COMMIT, "int eligible = (ttu <= ttr)", "int eligible = (ttu < ttr)"),
    ("commit_no_budget_check", COMMIT, "(claim_total_bytes <= budget_bytes) && ", ""),
    ("commit_new_vs_total", COMMIT, "(claim_new_bytes <= free_protected_bytes)", "(claim_total_bytes <= free_protected_bytes)"),
    ("commit_outcomes_swapped", COMMIT, "return retrieval_requested ? OR_ORDINARY : OR_BLOCKED;",
     "return retrieval_requested ? OR_BLOCKED : OR_ORDINARY;"),
    ("commit_request_not_eligible", COMMIT, "|| (retrieval_requested != 0)", ""),
    ("validate_reserved_ignored", VALIDATE, "if (jb->reserved != 0 || !or_job_ok(", "if (!or_job_ok("),
    ("validate_block_bound", VALIDATE, "if (blk < 0 || blk >= lo->num_blocks) return OR_VERANGE;",
     "if (blk < 0 || blk > lo->num_blocks) return OR_VERANGE;"),
    ("validate_job_compared_with_itself", VALIDATE, "for (int32_t p = 0; p < q; p++) {", "for (int32_t p = 0; p <= q; p++) {"),
    ("validate_within_job_unchecked", VALIDATE, "for (int32_t k = 0; k < i; k++)", "for (int32_t k = 0; k < 0; k++)"),
    ("validate_store_slots_unchecked", VALIDATE, "if (jobs[p].slot == jobs[q].slot) return OR_VEDUP;",
     "if (jobs[p].slot == jobs[q].slot && 0) return OR_VEDUP;"),
    ("validate_same_segment_only", VALIDATE,
     "== bt[(int64_t)jobs[p].req * bt_stride + (int64_t)jobs[p].chunk * nseg + k])",
     "== bt[(int64_t)jobs[p].req * bt_stride + (int64_t)jobs[p].chunk * nseg + i])"),
]

def _compile(src_text: str, out: str) -> None:
    c = out[:-3] + ".c"
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-w", "-o", out, c, "-lm"])


def _run_pins(lib_path: str, tests) -> subprocess.CompletedProcess:
    env = dict(os.environ, TEMPOKV_ORACLE_LIB=lib_path, HYPOTHESIS_PROFILE="default")
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-k", "not golden",
                           *tests], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


def test_unplanted_copy_passes_the_pins(tmp_path):
    # the harness itself: the oracle as committed, built the same way, passes every pin
    so = str(tmp_path / "liboracle_ref.so")
    _compile(open(SRC).read(), so)
    r = _run_pins(so, sorted(set(HASH + LOOKUP + COPY + COMMIT + VALIDATE)))
    assert r.returncode == 0, r.stdout[-3000:]


@pytest.mark.parametrize("name,tests,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, tests, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"{name}: the text to change must occur exactly once"
    so = str(tmp_path / f"liboracle_{name}.so")
    _compile(src.replace(old, new), so)
    r = _run_pins(so, tests)
    # exit 1: a pin failed; a negative code: the planted mistake crashed a pin run
    assert r.returncode == 1 or r.returncode < 0, f"{name} survived the pins:\n{r.stdout[-2000:]}"


# ---------------------------------------------------------------------------
# The controller oracle (plain Python): the same idea, the planted copy loaded
# in place of oracle.controller in a child process that runs its pin tests.
# ---------------------------------------------------------------------------
CTRL_SRC = os.path.join(ROOT, "oracle", "controller.py")
CTRL_PINS = ["tests/test_oracle_controller.py"]
_RUNNER = (
    "import sys, importlib.util\n"
    "import oracle\n"
    "spec = importlib.util.spec_from_file_location('oracle.controller', sys.argv[1])\n"
    "m = importlib.util.module_from_spec(spec)\n"
    "sys.modules['oracle.controller'] = m\n"
    "spec.loader.exec_module(m)\n"
    "oracle.controller = m\n"
    "import pytest\n"
    "sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', *sys.argv[2:]]))\n")

# Not listed: evaluating waiting claims before requested ones.  In this model every event gets its own
# control point and slots are filled greedily, so a claim becomes requested only at a control point where no
# other claim's eligibility or fit changed: the two orders decide the same, and no pin can tell them apart.
CTRL_MUTANTS = [
    ("shared_counted_twice", "            if prot[o] == 0:\n                P += obj_bytes[o]",
     "            if True:\n                P += obj_bytes[o]"),
    ("release_keeps_reservation", "                    if prot[o] == 0:\n                        P -= obj_bytes[o]",
     "                    if prot[o] == 0 and False:\n                        P -= obj_bytes[o]"),
    ("stage_reads_not_coalesced", "if not resident[o] and not queued[o]:\n                start", "if not resident[o]:\n                start"),
    ("state_ttr_ignores_queue", "    tail = max(busy_until, now)", "    tail = now"),
    ("state_ttr_first_object_decides", "            tail = tail + obj_bytes[o] / stage_rate\n            t_end = max(t_end, tail)",
     "            tail = tail + obj_bytes[o] / stage_rate\n            t_end = tail if t_end == now else t_end"),
    ("tempo_uses_static_ttr", "            ttu, ttr = (ttu_map[i] if i in ttu_map else math.inf), ttr_state(i)",
     "            ttu, ttr = (ttu_map[i] if i in ttu_map else math.inf), ttr_static(i)"),
    ("ttu_ignores_busy_slots", "        slots = [projected_end(a) for a in active] + [now] * (cfg.max_active - len(active))",
     "        slots = [now] * cfg.max_active"),
    ("ttu_counts_own_service", "            out[w] = s0 - now", "            out[w] = s0 + svc[w] - now"),
    ("queue_k_off_by_one", "(pos is not None and pos < cfg.queue_k)", "(pos is not None and pos <= cfg.queue_k)"),
    ("transfer_before_stage_ready", "            if state[i] == STAGEREADY:\n                state[i] = TRANSFERRING",
     "            if state[i] in (STAGEREADY, STAGING):\n                state[i] = TRANSFERRING"),
    ("release_at_request_end", "        elif kind == EV_TRANSFER_END:\n            if state[a] == TRANSFERRING:",
     "        elif kind == EV_TRANSFER_END:\n            if state[a] == TRANSFERRING and False:"),
    ("cost_not_per_request", "C=area / GIB / N", "C=area / GIB"),
    ("no_budget_headroom", "int(cfg.budget - P), int(new)", "int(cfg.budget), int(new)"),
    ("new_bytes_count_protected", "        new = sum(obj_bytes[o] for o in uniq[i] if prot[o] == 0)",
     "        new = sum(obj_bytes[o] for o in uniq[i])"),
    ("no_ticks", "            push((a + 1) * cfg.tick, EV_TICK, a + 1)", "            pass"),
    ("demand_commits_early", "            ttu, ttr = math.inf, 0.0\n        elif pol == IMMEDIATE:",
     "            ttu, ttr = 0.0, 0.0\n        elif pol == IMMEDIATE:"),
    ("ordinary_reads_free", "                fetch_end[i] = max(now, busy_until) + nonres / cfg.stage_rate",
     "                fetch_end[i] = now"),
    ("transfer_time_dropped", "                t_x = now + total[i] / cfg.gpu_rate\n                first_token[i]",
     "                t_x = now\n                first_token[i]"),
]


@pytest.mark.parametrize("name,old,new", CTRL_MUTANTS, ids=[m[0] for m in CTRL_MUTANTS])
def test_controller_pins_catch_planted_mistake(tmp_path, name, old, new):
    src = open(CTRL_SRC).read()
    assert src.count(old) == 1, f"{name}: the text to change must occur exactly once"
    path = tmp_path / "controller.py"
    path.write_text(src.replace(old, new))
    r = subprocess.run([sys.executable, "-c", _RUNNER, str(path), *CTRL_PINS], cwd=ROOT, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 1 or r.returncode < 0, f"{name} survived the pins:\n{r.stdout[-2000:]}"


def test_controller_unplanted_copy_passes_the_pins(tmp_path):
    path = tmp_path / "controller.py"
    path.write_text(open(CTRL_SRC).read())
    r = subprocess.run([sys.executable, "-c", _RUNNER, str(path), *CTRL_PINS], cwd=ROOT, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:]


# ---------------------------------------------------------------------------
# The oracle's commitment decisions over a batch of claims (oracle/pipeline.py):
# planted copies loaded in place of oracle.pipeline, against the closed-form
# pins of tests/test_claims.py (the "oracle_" tests).
# ---------------------------------------------------------------------------
PIPE_SRC = os.path.join(ROOT, "oracle", "pipeline.py")
_PIPE_RUNNER = _RUNNER.replace("oracle.controller", "oracle.pipeline").replace(
    "'-p', 'no:cacheprovider',", "'-p', 'no:cacheprovider', '-k', 'oracle_',")

PIPE_MUTANTS = [
    ("claims_in_request_order", "        order = [r for r in range(R) if requested[r]] + [r for r in range(R) if not requested[r]]",
     "        order = list(range(R))"),
    ("claims_shared_counted_twice", "            new = sum(slot_bytes for s in objs if s not in protected)",
     "            new = total"),
    ("claims_reservations_not_kept", "                reserved += new", "                reserved += 0"),
    ("claims_free_ignores_reservations", "            free = max(claims.budget_bytes - reserved, 0)",
     "            free = claims.budget_bytes"),
    ("claims_blocked_stops_walk", "            decision[r] = d\n", "            decision[r] = d\n            if d != oracle.COMMIT:\n                break\n"),
]


@pytest.mark.parametrize("name,old,new", PIPE_MUTANTS, ids=[m[0] for m in PIPE_MUTANTS])
def test_claim_pins_catch_planted_mistake(tmp_path, name, old, new):
    src = open(PIPE_SRC).read()
    assert src.count(old) == 1, f"{name}: the text to change must occur exactly once"
    path = tmp_path / "pipeline.py"
    path.write_text(src.replace(old, new))
    r = subprocess.run([sys.executable, "-c", _PIPE_RUNNER, str(path), "tests/test_claims.py"], cwd=ROOT,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 1 or r.returncode < 0, f"{name} survived the pins:\n{r.stdout[-2000:]}"


def test_claim_pins_pass_on_unplanted_copy(tmp_path):
    path = tmp_path / "pipeline.py"
    path.write_text(open(PIPE_SRC).read())
    r = subprocess.run([sys.executable, "-c", _PIPE_RUNNER, str(path), "tests/test_claims.py"], cwd=ROOT,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:]
