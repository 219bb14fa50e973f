"""Which bytes a warm request pre-reads into the caches (the cache touch), through the host
library: the extent minus a leading token-embedding table, for ResNet-50 and BERT models whose
span is 4 MB to 192 MB, never for an MLP. Byte counts from the models' layer tables."""
import pytest

import paper_2306_03622_amd as tp
import synth

MB = 1 << 20


def span(m):
    return tp.tph_touch_span(tp.ModelDesc.of(m), m.total_bytes, L=tp.host_lib())


def test_bert_base_skips_its_token_table():
    m = synth.config_model(4)
    tok = 30522 * 768 * 2                        # the leading token-embedding table
    assert m.total_bytes == 217_783_296
    assert span(m) == (tok, m.total_bytes)       # 170,901,504 bytes: within the 192 MB bound


def test_resnet50_touches_its_whole_extent():
    m = synth.config_model(3)
    assert span(m) == (0, m.total_bytes)


@pytest.mark.parametrize("cfg", [1, 2])
def test_mlps_are_never_touched(cfg):
    assert span(synth.config_model(cfg)) is None


def test_bounds_of_the_span():
    # a 2-layer BERT of width 64 is under 4 MB past its table; one of 8 layers of width 1024
    # (about 8 x 25 MB) is over 192 MB
    small = synth.bert(seed=1, layers=2, d=64, heads=1, ffn=256, seq=32, vocab=100, maxpos=32)
    assert small.total_bytes < 4 * MB and span(small) is None
    big = synth.bert(seed=2, layers=8, d=1024, heads=16, ffn=4096, seq=32, vocab=100, maxpos=32)
    assert big.total_bytes - 100 * 1024 * 2 > 192 * MB and span(big) is None
    mid = synth.bert(seed=3, layers=4, d=512, heads=8, ffn=2048, seq=64, vocab=1000, maxpos=64)
    lo, hi = span(mid)
    assert lo == -(-(1000 * 512 * 2) // 256) * 256 and hi == mid.total_bytes
