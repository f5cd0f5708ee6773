"""The oracle against its pins (CPU only)."""

import pytest

import oracle_checks as C


def test_prefill_golden():
    C.check_prefill_golden()


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("per_chunk", [False, True])
def test_prefill_blockdiag_bruteforce(seed, per_chunk):
    C.check_prefill_blockdiag_bruteforce(seed, per_chunk)


@pytest.mark.parametrize("seed", [3, 4])
def test_prefill_sdpa(seed):
    C.check_prefill_sdpa(seed)


def test_prefill_q_zero():
    C.check_prefill_q_zero(5)


def test_prefill_v_const():
    C.check_prefill_v_const(6)


def test_prefill_rowsums():
    C.check_prefill_rowsums(7)


def test_cache_exact():
    C.check_cache_exact(8)


def test_key_mean_const():
    C.check_key_mean_const(9)


def test_select_golden():
    C.check_select_golden()


def test_chunk_score_zero_query():
    C.check_chunk_score_zero_query(10)


def test_chunk_score_linear():
    C.check_chunk_score_linear(11)


def test_chunk_score_gqa_groups():
    C.check_chunk_score_gqa_groups(12)


def test_topk_bruteforce():
    C.check_topk_bruteforce(13)


def test_token_rank():
    C.check_token_rank(16)


def test_decode_golden():
    C.check_decode_golden()


@pytest.mark.parametrize("n_static", [0, 2, 4])
def test_decode_dense(n_static):
    C.check_decode_dense(14, n_static)


def test_decode_permutation():
    C.check_decode_permutation(15)


def test_static_golden():
    C.check_static_golden()


@pytest.mark.parametrize("seed", [1, 2])
def test_gather_matches_decode_rows(seed):
    C.check_gather_matches_decode_rows(seed)


@pytest.mark.parametrize("n_static", [0, 3])
def test_compact_decode_equals_gathered(n_static):
    C.check_compact_decode_equals_gathered(7, n_static)


def test_compact_decode_sdpa():
    C.check_compact_decode_sdpa(5)


def test_chunk_score_golden():
    C.check_chunk_score_golden()


@pytest.mark.parametrize("m_len", [0, 4])
def test_chunk_score_uniform(m_len):
    C.check_chunk_score_uniform(21, m_len)


@pytest.mark.parametrize("seed", [22, 23])
def test_chunk_score_bruteforce(seed):
    C.check_chunk_score_bruteforce(seed)


def test_select_ranked_bruteforce():
    C.check_select_ranked_bruteforce(24)


def test_full_mask_golden():
    C.check_full_mask_golden()


def test_rope_composition():
    C.check_rope_composition(31)


@pytest.mark.parametrize("seed", [32, 33])
def test_joint_rows(seed):
    C.check_joint_rows(seed)


def test_joint_attention_sdpa():
    C.check_joint_attention_sdpa(34)


def test_full_mask_dense():
    C.check_full_mask_dense(35)
