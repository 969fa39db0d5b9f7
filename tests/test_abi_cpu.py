"""The C-ABI library loads without a GPU, exports every symbol the header
declares, sizes workspaces, and rejects bad arguments on the host before
enqueueing anything (CPU only; no compute call)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "luffy.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2411_15419_amd as L
    if not os.path.exists(L.LIB_PATH):
        from paper_2411_15419_amd import build
        build.build()
    return L.load_library()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(luffy_[a-z_]+)\s*\(", text)))


def test_header_lists_the_four_calls():
    names = header_functions()
    for n in ("luffy_route", "luffy_condense", "luffy_expert_ffn", "luffy_combine"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in header_functions():
        assert hasattr(lib, name), name


def test_version_and_strings(lib):
    assert lib.luffy_abi_version() == 6
    assert lib.luffy_status_string(0) == b"ok"
    assert lib.luffy_status_string(-3).startswith(b"workspace")


def test_capacity_agrees_with_the_oracle(lib):
    """luffy_capacity (what luffy_route drops at, and what MoELayer sizes
    max_bucket from) equals the oracle's capacity_of on a grid that includes
    decimal factors whose product with k*T/E is an integer (cf = 1.1 with
    k*T/E = 1000: a float32 factor would give 1101)."""
    from oracle import luffy_oracle as O
    import paper_2411_15419_amd as L
    assert lib.luffy_capacity(4000, 2, 8, 1.1) == 1100
    assert O.capacity_of(4000, 2, 8, 1.1) == 1100
    for T in (1, 7, 1000, 4000, 8192, 32768, 65536):
        for k in (1, 2):
            for E in (1, 3, 8, 16, 64):
                for cf in (0.0, -1.0, 0.1, 0.3, 0.75, 1.0, 1.1, 1.2, 1.25, 1.3, 2.0, 2.5):
                    assert lib.luffy_capacity(T, k, E, cf) == O.capacity_of(T, k, E, cf), (T, k, E, cf)
                    assert L.capacity(T, k, E, cf) == O.capacity_of(T, k, E, cf)


def test_workspace_sizes(lib):
    import paper_2411_15419_amd as L
    assert L.route_workspace_size(8192, 16, 2) >= 16 * 16 * 4
    # bitmask: T*k rows of ceil(max_bucket/64) words
    c3 = L.condense_workspace_size(32768, 2048, 32, 2, 32768)
    assert c3 >= 65536 * 512 * 8
    assert L.condense_workspace_size(65536, 1024, 64, 1, 1024) < c3
    assert L.expert_ffn_workspace_size(65536, 32, 8192, L.LUFFY_BF16) >= 65536 * 8192 * 2
    assert L.route_workspace_size(0, 16, 2) == 0


def test_invalid_arguments_rejected_on_host(lib):
    fake = ctypes.c_void_p(256)     # never dereferenced: validation fails first
    # null pointers
    assert lib.luffy_route(None, 8, 64, 1, fake, None, 4, 1, 0.0, fake, fake, fake, fake,
                           fake, None, fake, 1 << 20, None) == -1
    # k out of range, k > E
    assert lib.luffy_route(fake, 8, 64, 1, fake, None, 4, 3, 0.0, fake, fake, fake, fake,
                           fake, None, fake, 1 << 20, None) == -1
    assert lib.luffy_route(fake, 8, 64, 1, fake, None, 1, 2, 0.0, fake, fake, fake, fake,
                           fake, None, fake, 1 << 20, None) == -1
    # unsupported sizes
    assert lib.luffy_route(fake, 8, 65, 1, fake, None, 4, 1, 0.0, fake, fake, fake, fake,
                           fake, None, fake, 1 << 20, None) == -2
    assert lib.luffy_route(fake, 8, 64, 1, fake, None, 65, 1, 0.0, fake, fake, fake, fake,
                           fake, None, fake, 1 << 20, None) == -2
    # workspace too small / misaligned
    assert lib.luffy_route(fake, 8, 64, 1, fake, None, 4, 1, 0.0, fake, fake, fake, fake,
                           fake, None, fake, 0, None) == -3
    assert lib.luffy_route(fake, 8, 64, 1, fake, None, 4, 1, 0.0, fake, fake, fake, fake,
                           fake, None, ctypes.c_void_p(260), 1 << 20, None) == -3
    assert b"workspace" in lib.luffy_last_error()
    # condense: NaN threshold, bad dtype
    assert lib.luffy_condense(fake, 8, 64, 1, fake, fake, 4, 1, 8, float("nan"), fake, fake,
                              fake, fake, None, None, None, fake, 1 << 30, None) == -1
    assert lib.luffy_condense(fake, 8, 64, 7, fake, fake, 4, 1, 8, 0.9, fake, fake,
                              fake, fake, None, None, None, fake, 1 << 30, None) == -1
    # ffn: unknown activation, d_ff not a multiple of 64
    assert lib.luffy_expert_ffn(fake, None, fake, 4, 64, 128, 1, fake, fake, 9, 8, fake,
                                fake, 1 << 30, None) == -1
    assert lib.luffy_expert_ffn(fake, None, fake, 4, 64, 100, 1, fake, fake, 0, 8, fake,
                                fake, 1 << 30, None) == -2
    # combine: k not 1/2
    assert lib.luffy_combine(fake, fake, fake, fake, 8, 3, 64, 1, fake, None) == -1
    # combine backward: null pointer, k not 1/2, d not a multiple of 64, workspace too small
    assert lib.luffy_combine_backward(None, fake, fake, fake, fake, fake, fake, fake, 4, 8, 2, 64, 1, 16,
                                      fake, fake, fake, 1 << 20, None) == -1
    assert lib.luffy_combine_backward(fake, fake, fake, fake, fake, fake, fake, fake, 4, 8, 3, 64, 1, 16,
                                      fake, fake, fake, 1 << 20, None) == -1
    assert lib.luffy_combine_backward(fake, fake, fake, fake, fake, fake, fake, fake, 4, 8, 2, 96, 1, 16,
                                      fake, fake, fake, 1 << 20, None) == -2
    assert lib.luffy_combine_backward(fake, fake, fake, fake, fake, fake, fake, fake, 4, 8, 2, 64, 1, 16,
                                      fake, fake, fake, 16, None) == -3
    # expert FFN backward: bf16 only, unknown activation, unknown weight-
    # gradient dtype, workspace too small (with either gradient dtype)
    assert lib.luffy_expert_ffn_backward(fake, None, fake, 4, 64, 128, 0, fake, fake, 0, 8, fake, fake,
                                         fake, fake, 0, fake, 1 << 30, None) == -2
    assert lib.luffy_expert_ffn_backward(fake, None, fake, 4, 64, 128, 1, fake, fake, 9, 8, fake, fake,
                                         fake, fake, 0, fake, 1 << 30, None) == -1
    assert lib.luffy_expert_ffn_backward(fake, None, fake, 4, 64, 128, 1, fake, fake, 0, 8, fake, fake,
                                         fake, fake, 2, fake, 1 << 30, None) == -1
    for dw in (0, 1):
        assert lib.luffy_expert_ffn_backward(fake, None, fake, 4, 64, 128, 1, fake, fake, 0, 8, fake, fake,
                                             fake, fake, dw, fake, 256, None) == -3
    assert lib.luffy_expert_ffn_backward_workspace_size(8, 4, 64, 128, 0) == 0   # float32: none


def test_history_record_layout(lib):
    """luffy_history_size is the record layout the header documents:
    sections info[8] int32, slot_pos[T*k] int32, offsets[E+1] int32,
    word_off[E+1] int64, hi[W] and lo[W] uint64 with W = T*k*ceil(max_bucket/64),
    each starting at a multiple of 256 bytes."""
    def up(v):
        return (v + 255) // 256 * 256
    for T, E, k, mb in ((2048, 8, 2, 2048), (512, 4, 1, 512), (65536, 64, 1, 1024), (32768, 32, 2, 32768)):
        W = T * k * ((mb + 63) // 64)
        size = 0
        for nbytes in (32, 4 * T * k, 4 * (E + 1), 8 * (E + 1), 8 * W, 8 * W):
            size = up(size) + nbytes
        assert lib.luffy_history_size(T, E, k, mb) == up(size), (T, E, k, mb)
    assert lib.luffy_condense_history_workspace_size(2048, 256, 8, 2, 2048) > \
        lib.luffy_condense_workspace_size(2048, 256, 8, 2, 2048)


def test_history_arguments_rejected_on_host(lib):
    fake = ctypes.c_void_p(256)
    args = [fake, 8, 64, 1, fake, fake, fake, 4, 1, 8, 0.9, None, None, 0.8, 0.2, fake, fake, fake, fake,
            None, None, None, None, fake, 1 << 30, None]
    ok_ws = lib.luffy_condense_history_workspace_size(8, 64, 4, 1, 8)
    assert ok_ws > 0
    def call(**kw):
        a = list(args)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return lib.luffy_condense_history(*a)
    assert call(a0=None) == -1                       # null x
    assert call(a13=float("nan")) == -1              # S1 NaN
    assert call(a12=fake, a6=None) == -1             # hist_out without slot_pos
    assert call(a11=fake, a12=fake) == -1            # hist_in aliases hist_out
    assert call(a11=ctypes.c_void_p(260)) == -1      # misaligned record
    assert call(a24=16) == -3                        # workspace too small


def test_binding_refuses_cpu_tensors(lib):
    import torch
    import paper_2411_15419_amd as L
    x = torch.zeros(8, 64, dtype=torch.bfloat16)
    with pytest.raises(L.LuffyError):
        L.luffy_combine(x, torch.zeros(8, dtype=torch.int32), torch.zeros(8, 1, dtype=torch.int32),
                        torch.zeros(8, 1), x)
