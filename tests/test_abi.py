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


def _entry_calls(pbg, ctx):
    """Every entry point that takes a context, called on ctx with empty
    arguments (nothing that a check would let reach a device)."""
    import ctypes
    neg = pbg.NegConfig(1, 1, 1, 0, 0)
    d = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    st = pbg.Stats()
    return {
        "pbg_bucket_edges": (ctx, None, None, None, 0, None, None, None, None),
        "pbg_bind_partition": (ctx, 0, None, None, 0),
        "pbg_bind_relations": (ctx, None, None),
        "pbg_set_streams": (ctx, None, None),
        "pbg_train_bucket": (ctx, 0, 0, None, None, None, 0, ctypes.byref(neg), 0.1, 1, ctypes.byref(d)),
        "pbg_set_entity_types": (ctx, 1, None, None, None, None),
        "pbg_bind_type_partition": (ctx, 0, 0, None, None, 0),
        "pbg_set_relation_weights": (ctx, None),
        "pbg_group_by_relation": (ctx, None, None, None, 0, None, None, None),
        "pbg_get_step_losses": (ctx, None, 0, ctypes.byref(n)),
        "pbg_train_epoch": (ctx, None, None, None, None, ctypes.byref(neg), 0.1, 1, 1, ctypes.byref(d)),
        "pbg_score_edges": (ctx, 0, 0, None, None, None, 0, None),
        "pbg_score_edges_noalloc": (ctx, 0, 0, None, None, None, 0, None),
        "pbg_rank_eval": (ctx, None, None, None, 0, None, None, None, 0, None, ctypes.byref(d), ctypes.byref(d)),
        "pbg_rank_sampled": (ctx, None, None, None, 0, None, 0, None, ctypes.byref(d), ctypes.byref(d)),
        "pbg_sample_negatives": (ctx, 0, 0, 0, 0, 1, 1, None),
        "pbg_inspect_step": (ctx, 0, 0, None, None, None, 0, ctypes.byref(neg), 1, None, None, None, None,
                             ctypes.byref(d)),
        "pbg_get_stats": (ctx, ctypes.byref(st)),
    }


def test_every_entry_point_rejects_a_null_context():
    """Sec. 4 runtime boundary: a NULL context is an argument error for every
    call, the queries answer -1, and freeing it does nothing."""
    from paper_1903_12287_amd import pbg
    if not os.path.exists(pbg.LIB_PATH):
        pytest.skip("library not built")
    lib = pbg.library()
    calls = _entry_calls(pbg, None)
    # every declared entry point is either here or one of the non-status calls
    others = {"pbg_bucket_init", "pbg_free", "pbg_last_error", "pbg_partition_rows", "pbg_relation_param_floats",
              "pbg_type_partition_rows"}
    assert sorted(set(calls) | others) == _declared()
    for name, args in calls.items():
        assert getattr(lib, name)(*args) == 1, name   # PBG_ERR_INVALID_ARG
    assert lib.pbg_partition_rows(None, 0) == -1
    assert lib.pbg_type_partition_rows(None, 0, 0) == -1
    assert lib.pbg_relation_param_floats(None) == -1
    assert lib.pbg_last_error(None)
    lib.pbg_free(None)
    import ctypes
    assert lib.pbg_bucket_init(None, 10, 1, 1, 8, 0, 0, 0, 0.1, 0) == 1
    ctx = ctypes.c_void_p()
    assert lib.pbg_bucket_init(ctypes.byref(ctx), 10, 1, 1, 8, 0, 0, 0, 0.1, 1 << 20) == 1   # unknown flag
    assert ctx.value and b"flags" in lib.pbg_last_error(ctx)
    lib.pbg_free(ctx)


def test_a_context_that_failed_to_initialise_rejects_every_call():
    """Wrong call order: a context whose initialisation failed is kept only
    to carry its message; every other call reports a state error."""
    import ctypes
    from paper_1903_12287_amd import pbg
    if not os.path.exists(pbg.LIB_PATH):
        pytest.skip("library not built")
    lib = pbg.library()
    ctx = ctypes.c_void_p()
    assert lib.pbg_bucket_init(ctypes.byref(ctx), 10, 1, 1, 0, 0, 0, 0, 0.1, 0) == 1   # dim 0
    assert ctx.value
    msg = lib.pbg_last_error(ctx)
    try:
        for name, args in _entry_calls(pbg, ctx).items():
            assert getattr(lib, name)(*args) == 5, name   # PBG_ERR_STATE
        assert lib.pbg_partition_rows(ctx, 0) == -1
        assert lib.pbg_type_partition_rows(ctx, 0, 0) == -1
        assert lib.pbg_relation_param_floats(ctx) == -1
    finally:
        lib.pbg_free(ctx)
    assert b"dim" in msg
