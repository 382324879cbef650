"""The C-ABI library loads and exports every entry point that include/pbg.h
declares; argument errors are reported without a device (no compute calls)."""

import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pbg.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)   # declarations only, not comments
    return sorted(set(re.findall(r"\b(pbg_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    for want in ("pbg_bucket_init", "pbg_train_bucket", "pbg_score_edges", "pbg_rank_eval", "pbg_rank_sampled",
                 "pbg_bucket_edges", "pbg_train_epoch", "pbg_bind_partition"):
        assert want in names


def test_library_exports_every_declared_symbol():
    from paper_1903_12287_amd import pbg
    if not os.path.exists(pbg.LIB_PATH):
        pytest.skip("library not built")
    lib = pbg.library()
    for name in _declared():
        assert hasattr(lib, name), name
    assert sorted(pbg.EXPORTS) == _declared()


def test_init_rejects_bad_arguments_without_a_device():
    from paper_1903_12287_amd import pbg
    if not os.path.exists(pbg.LIB_PATH):
        pytest.skip("library not built")
    bad = [
        dict(num_entities=0, num_partitions=1, num_relations=1, dim=8, op=0, cmp=0, loss=0),
        dict(num_entities=10, num_partitions=1, num_relations=1, dim=0, op=0, cmp=0, loss=0),
        dict(num_entities=10, num_partitions=1, num_relations=1, dim=513, op=0, cmp=0, loss=0),
        dict(num_entities=10, num_partitions=1, num_relations=1, dim=7, op=4, cmp=0, loss=0),
        dict(num_entities=10, num_partitions=1, num_relations=1, dim=8, op=9, cmp=0, loss=0),
        dict(num_entities=10, num_partitions=1, num_relations=1, dim=8, op=0, cmp=5, loss=0),
        dict(num_entities=10, num_partitions=1, num_relations=1, dim=8, op=0, cmp=0, loss=7),
        dict(num_entities=9, num_partitions=4, num_relations=1, dim=8, op=0, cmp=0, loss=0),
    ]
    for kw in bad:
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_bucket_init(kw["num_entities"], kw["num_partitions"], kw["num_relations"],
                                kw["dim"], kw["op"], kw["cmp"], kw["loss"])
        assert ei.value.status_name == "INVALID_ARG", kw
    with pytest.raises(pbg.PbgError) as ei:
        pbg.pbg_bucket_init(100, 1, 3, 8, "linear", "cos", "ranking")
    assert ei.value.status_name == "UNSUPPORTED"
