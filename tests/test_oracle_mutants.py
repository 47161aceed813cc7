"""The pins must catch plausible mistakes: each mutant below plants one in a
copy of the oracle's C source (on the CPU, in a temporary directory), and the
pin suite, pointed at the mutant library, must fail."""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

MUTANTS = {
    "copy starts one after the neighbour": ("int64_t p = (int64_t)i + 1 + m;", "int64_t p = (int64_t)i + m;"),
    "trace boundary ignored": ("if (p >= n_valid || traces[p] != traces[i])", "if (p >= n_valid)"),
    "band edge exclusive": ("if (sc >= band_min[j]) {", "if (sc > band_min[j]) {"),
    "theta exclusive": ("if (best >= theta)", "if (best > theta)"),
    "short chains kept": ("if (got < 2) {", "if (got < 1) {"),
    "ties broken by higher index": ("return (a->i < b->i) ? -1 : (a->i > b->i);", "return (a->i > b->i) ? -1 : (a->i < b->i);"),
    "lexical budget rolls over": ("        spent = 0;\n        for (int32_t c = 0; c < k; c++) {", "        spent = spent - lex_budget;\n        for (int32_t c = 0; c < k; c++) {"),
    "root charged to the budget": ("        int32_t count = 0, spent = 0;", "        int32_t count = 0, spent = 1;"),
    "no prefix walk (root-attached)": ("        orc_node *next = find_child(cur, chain[m]);", "        orc_node *next = m < 0 ? find_child(cur, chain[m]) : NULL;"),
    "norm without square root": ("double norm = sqrt(ss);", "double norm = ss;"),
    "rounding ties away from zero": ("pick = (fmod(fabs(lo), 2.0) == 0.0) ? lo : hi;", "pick = hi;"),
    "score drops the last dim": ("for (int32_t j = 0; j < d; j++)\n                acc +=", "for (int32_t j = 0; j < d - 1; j++)\n                acc +="),
    "exclusion ignored": ("if (prompt && exclude && exclude[b] >= 0 && prompt[i] == exclude[b])", "if (0)"),
    "mask misses the node itself": ("            int32_t j = i, guard = 0;", "            int32_t j = node_parent[(int64_t)b * max_nodes + i], guard = 0;"),
    "bonus always from the root": ("        bonus[b] = target[o + cur];", "        bonus[b] = target[o];"),
    "suffix match crosses traces": ("p - m >= 0 && lv_same_trace(v, p - m, p) && lv_tok", "p - m >= 0 && lv_tok"),
    "draft starts at the match": ("ot[(int64_t)n_picked * L_lex + j] = lv_tok(v, p + 1 + j);", "ot[(int64_t)n_picked * L_lex + j] = lv_tok(v, p + j);"),
    "rarest continuation first": ("return a->count > b->count ? -1 : 1;", "return a->count < b->count ? -1 : 1;"),
    "lexical ties by latest position": ("return (a->p < b->p) ? -1 : (a->p > b->p);", "return (a->p > b->p) ? -1 : (a->p < b->p);"),
    "lexical self-exclusion ignored": ("(p < n_valid && ex >= 0 && prompts[p] == ex)", "(0)"),
    "draft not clipped at trace end": ("p + 1 + len < end && lv_same_trace(v, p + 1 + len, p)", "p + 1 + len < end"),
    "history ignored": ("            view.hl = hl;", "            view.hl = 0;"),
    "history joined to the store's last trace": ("    return p >= v->n_valid && q >= v->n_valid;", "    return 1;"),
    "history removed by self-exclusion": ("(p < n_valid && ex >= 0 && prompts[p] == ex)", "(ex >= 0 && (p >= n_valid || prompts[p] == ex))"),
    "every request sees the first history": ("view.hist = hist + (int64_t)b * H;", "view.hist = hist;"),
    "history read one token past its length": ("            view.hl = hl;", "            view.hl = hl < H ? hl + 1 : hl;"),
    "overlong history dropped instead of cut": ("(hist_len[b] > H ? H : hist_len[b])", "(hist_len[b] > H ? 0 : hist_len[b])"),
    "capacity ignored": ("if (n_ge + n_at[m] > max_cand)", "if (0)"),
    "held draft proposed again": ("if (picked[t] == g)", "if (picked[t] == -7)"),
    "accepted nodes recycled too": ("            if (accepted[n])\n                continue;", "            if (0)\n                continue;"),
    "record keyed by the node's own state": ("rec_src[k] = (int32_t)(o + parent);", "rec_src[k] = (int32_t)(o + n);"),
    "rollout skips the node's own prediction": ("            out[len++] = target[o + cur];\n            while (len < depth) {", "            while (len < depth) {"),
    "rollout one deeper": ("            while (len < depth) {", "            while (len <= depth) {"),
    "recycled lookup ignores the token": ("            if (tokens[r] != anchor[b])\n                continue;", "            if (0)\n                continue;"),
    "recycled threshold exclusive": ("            if ((float)acc < theta)", "            if ((float)acc <= theta)"),
    "recycled score drops the last dim": ("for (int32_t e = 0; e < d; e++)", "for (int32_t e = 0; e < d - 1; e++)"),
    "rollouts under their own budget": ("            insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 3,", "            spent = 0;\n            insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 3,"),
    "e4m3 ties away from zero": ("        pick = (fmod(q, 2.0) == 0.0) ? lo : hi; /* tie: the even multiple */", "        pick = hi;"),
    "e4m3 exponent bias 8": ("        v = ldexp(1.0 + (double)m / 8.0, e - 7);", "        v = ldexp(1.0 + (double)m / 8.0, e - 8);"),
    "fp8 scale one binade up": ("int shift = m > 0.0 ? 7 - e : 0;", "int shift = m > 0.0 ? 8 - e : 0;"),
    "e4m3 subnormal spacing halved": ("        spacing = ldexp(1.0, -9);", "        spacing = ldexp(1.0, -10);"),
    "fp8 score drops the query scale": ("s[(int64_t)b * n + i] = acc * kinv[i] * qinv[b];", "s[(int64_t)b * n + i] = acc * kinv[i];"),
    "fp8 score drops the last dim": ("            for (int32_t c = 0; c < d; c++)\n                acc += kv[c]", "            for (int32_t c = 0; c < d - 1; c++)\n                acc += kv[c]"),
    "lexical branches left out of C": ("        for (int32_t c = 0; c < n_lex_ret; c++) {", "        for (int32_t c = 0; c < 0; c++) {"),
    "lexical branches not cut to their limit": ("            if (len > L_lex_ret)\n                len = L_lex_ret;", "            if (0)\n                len = L_lex_ret;"),
    "lexical branch nodes tagged as the allocation's": ("insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 4,", "insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 1,"),
    "every lexical draft joins C": ("    if (n_lex_ret > n_lex)\n        n_lex_ret = n_lex;", "    if (1)\n        n_lex_ret = n_lex;"),
    "lexical branches before the retrieved chains": (
        "        for (int32_t c = 0; c < k; c++) {\n            int64_t o = (int64_t)b * k + c;\n"
        "            int32_t len = sem_len[o] < L ? sem_len[o] : L;\n"
        "            insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 2, sem_tokens + o * L, len);\n"
        "        }\n"
        "        /* the top lexical branches join C after the retrieved chains (Algorithm 1,\n"
        "           lexical step), cut to L_lex_ret tokens */\n"
        "        for (int32_t c = 0; c < n_lex_ret; c++) {",
        "        for (int32_t c = 0; c < n_lex_ret; c++) {\n"
        "            int64_t o = (int64_t)b * n_lex + c;\n"
        "            int32_t len = lex_len[o] < L_lex ? lex_len[o] : L_lex;\n"
        "            if (len > L_lex_ret)\n                len = L_lex_ret;\n"
        "            insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 4, lex_tokens + o * L_lex, len);\n"
        "        }\n"
        "        for (int32_t c = 0; c < k; c++) {\n            int64_t o = (int64_t)b * k + c;\n"
        "            int32_t len = sem_len[o] < L ? sem_len[o] : L;\n"
        "            insert_chain(nodes, &count, max_nodes, &spent, sem_budget, 2, sem_tokens + o * L, len);\n"
        "        }\n"
        "        for (int32_t c = 0; c < 0; c++) {"),
    "capacity flag misses an overflowing longest level": ("out_capped[b] = (n_at[mtop] > max_cand || (cut_below", "out_capped[b] = (0 || (cut_below"),
    "capacity flag ignores how many drafts are held": ("(cut_below && n_picked < n_lex)) ? 1 : 0;", "(cut_below)) ? 1 : 0;"),
    "recycled ties by newest": ("    return (a->seq < b->seq) ? -1 : (a->seq > b->seq);", "    return (a->seq > b->seq) ? -1 : (a->seq < b->seq);"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name!r} not found exactly once"
    with tempfile.TemporaryDirectory() as td:
        c = os.path.join(td, "mut.c")
        so = os.path.join(td, "libmut.so")
        open(c, "w").write(src.replace(old, new))
        subprocess.run(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC",
                        "-shared", "-std=c11", "-o", so, c, "-lm"], check=True)
        env = dict(os.environ, OILBIRD_ORACLE_LIB=so)
        r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                            os.path.join(ROOT, "tests", "test_oracle.py"),
                            os.path.join(ROOT, "tests", "test_oracle_verify.py"),
                            os.path.join(ROOT, "tests", "test_oracle_lexical.py"),
                            os.path.join(ROOT, "tests", "test_oracle_recycle.py"),
                            os.path.join(ROOT, "tests", "test_oracle_fp8.py")],
                           env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
        assert r.returncode != 0, f"pins did not catch mutant {name!r}"
