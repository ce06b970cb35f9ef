"""The exported C ABI against the boundary the hot path was specified with: every entry
point's parameters, parsed from include/packmamba.h, are the specified ones in the
specified order, plus only the documented insertions (each with its reason), so that a
caller of the specified interface finds every argument where it expects it relative
to the others.  CPU only."""
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "packmamba.h")

STATES = "per-row initial/final states and their gradients (state passing across rows)"
# name: (specified parameters in order, {inserted parameter: (the parameter it follows, reason)})
SPEC = {
    "packmamba_causal_conv1d_fwd": (
        ["x", "weight", "bias", "position_indices", "out", "batch", "dim", "seqlen", "width", "dtype", "silu",
         "stream"],
        {"initial_x": ("position_indices", STATES), "final_x": ("out", STATES)}),
    "packmamba_causal_conv1d_bwd": (
        ["x", "weight", "bias", "position_indices", "dout", "dx", "dweight", "dbias", "workspace",
         "workspace_bytes", "batch", "dim", "seqlen", "width", "dtype", "silu", "stream"],
        {"initial_x": ("position_indices", STATES), "dfinal_x": ("dout", STATES),
         "dinitial_x": ("dbias", STATES)}),
    "packmamba_selective_scan_fwd": (
        ["u", "delta", "A", "B", "C", "D", "z", "delta_bias", "delta_softplus", "position_indices", "out",
         "saved_states", "batch", "dim", "seqlen", "dstate", "dtype", "stream"],
        {"initial_state": ("position_indices", STATES), "final_state": ("out", STATES),
         "workspace": ("saved_states", "segment carries when long rows are split across blocks"),
         "workspace_bytes": ("workspace", "size of that workspace")}),
    "packmamba_selective_scan_bwd": (
        ["u", "delta", "A", "B", "C", "D", "z", "delta_bias", "delta_softplus", "position_indices", "dout",
         "saved_states", "du", "ddelta", "dA", "dB", "dC", "dD", "dz", "ddelta_bias", "workspace",
         "workspace_bytes", "batch", "dim", "seqlen", "dstate", "dtype", "stream"],
        {"initial_state": ("position_indices", STATES), "dfinal_state": ("dout", STATES),
         "dinitial_state": ("ddelta_bias", STATES)}),
    "packmamba_selective_scan_fwd_saved_states_size": (["batch", "dim", "seqlen", "dstate"], {}),
    "packmamba_selective_scan_bwd_workspace_size": (["batch", "dim", "seqlen", "dstate"], {}),
    "packmamba_causal_conv1d_bwd_workspace_size": (["batch", "dim", "seqlen", "width"], {}),
    "packmamba_check_position_indices": (
        ["position_indices", "batch", "seqlen", "d_flag", "stream"],
        {"continued": ("seqlen", "rows may start inside a sequence continued from another row")}),
    "packmamba_status_string": (["status"], {}),
    "packmamba_abi_version": ([], {}),
}
# entry points beyond the specified boundary, with the reason they exist
ADDED = {
    "packmamba_selective_scan_fwd_workspace_size": "size of the forward's segment workspace",
    "packmamba_rmsnorm_fwd": "packed Mamba block: RMSNorm forward",
    "packmamba_rmsnorm_bwd": "packed Mamba block: RMSNorm backward",
    "packmamba_rmsnorm_bwd_workspace_size": "packed Mamba block: RMSNorm backward workspace",
    "packmamba_pack_plan": "host packing policies",
    "packmamba_pack_positions": "host packing policies",
    "packmamba_causal_conv1d_bwd_noalloc": "conv backward for callers that cannot allocate",
}


def parse_header():
    """{function name: [parameter names]} of every declaration in the header."""
    text = re.sub(r"/\*.*?\*/", " ", open(HEADER).read(), flags=re.S)
    out = {}
    for m in re.finditer(r"\b(packmamba_\w+)\s*\(([^;{]*?)\)\s*;", text):
        params = [p.strip() for p in m.group(2).split(",") if p.strip() and p.strip() != "void"]
        out[m.group(1)] = [re.findall(r"\w+", p)[-1] for p in params]
    return out


def expected(spec, inserted):
    order = list(spec)
    pending = dict(inserted)
    while pending:
        progressed = False
        for name, (after, _) in list(pending.items()):
            if after in order:
                order.insert(order.index(after) + 1, name)
                del pending[name]
                progressed = True
        assert progressed, pending
    return order


def test_every_specified_entry_point_keeps_its_order():
    got = parse_header()
    for name, (spec, inserted) in SPEC.items():
        assert name in got, name
        assert got[name] == expected(spec, inserted), (name, got[name])
        # removing the documented insertions gives back the specified list exactly
        assert [p for p in got[name] if p not in inserted] == spec, name


def test_no_undocumented_entry_points():
    got = parse_header()
    assert set(got) == set(SPEC) | set(ADDED), set(got) ^ (set(SPEC) | set(ADDED))


def test_stream_is_an_opaque_pointer_and_dtype_codes():
    """The stream is passed as void* (a hipStream_t) so that the header needs no HIP
    include; the dtype codes are the specified two plus bf16 inputs with fp32 outputs."""
    text = open(HEADER).read()
    assert "#include <hip" not in text
    for name in ("packmamba_causal_conv1d_fwd", "packmamba_selective_scan_bwd"):
        decl = re.search(name + r"\s*\(([^;]*?)\)\s*;", re.sub(r"/\*.*?\*/", " ", text, flags=re.S)).group(1)
        assert re.search(r"void\s*\*\s*stream\s*$", decl.strip()), name
    codes = dict(re.findall(r"#define (PACKMAMBA_(?:F32|BF16|BF16_F32OUT)) (\d+)", text))
    assert codes == {"PACKMAMBA_F32": "0", "PACKMAMBA_BF16": "1", "PACKMAMBA_BF16_F32OUT": "2"}
