"""Distance, in wait states, from each matrix-core (XDL) instruction of the partial kernel to the
first later instruction that reads a register it wrote, in the AMD assembly of this build.

An XDL op's result is written back some cycles after issue; an instruction that reads the result
earlier sees the old register contents.  The toolchain pads such reads to its own model of the
op (8 wait states for v_mfma_f32_16x16x32_bf16 on gfx950: a 4-pass op, passes + 3 + 1).  With
only that padding the kernel's first reads of the q.k scores were seen to return the previous
slice's scores, so the kernel adds 16 more there (xdl_result_wait).  This scan checks, kernel by
kernel, that every read of an XDL result by a vector, LDS or memory instruction along the
fall-through path is at least MIN_WAIT states after the op (an XDL op accumulating onto the result
is forwarded inside the matrix core and is not counted).  Counting: s_nop N is N + 1 states, any other instruction 1; a register rewritten
before it is read no longer holds the result."""
import re
import subprocess

MIN_WAIT = 16


def _regs(tok):
    tok = tok.strip().rstrip(",")
    m = re.match(r"^([va])\[(\d+):(\d+)\]$", tok)
    if m:
        return {f"{m.group(1)}{i}" for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"^([va])(\d+)$", tok)
    return {tok} if m else set()


def _operands(ins):
    parts = ins.split(None, 1)
    return parts[0], (parts[1].split(", ") if len(parts) > 1 else [])


def _writes(op, ops):
    if op.startswith(("v_", "ds_read", "buffer_load", "global_load", "scratch_load")) and ops:
        if op.startswith(("v_cmp", "v_cmpx")) and not op.endswith("_e64"):
            return set()
        return _regs(ops[0])
    return set()


def _reads(op, ops):
    if op.startswith(("v_", "ds_", "buffer_", "global_", "scratch_")):
        dst_first = op.startswith(("v_", "ds_read", "buffer_load", "global_load", "scratch_load"))
        out = set()
        for t in (ops[1:] if dst_first else ops):
            out |= _regs(t)
        return out
    return set()


def scan(asm: str, kernel: str, horizon: int = 120):
    """(wait states, op index, reader index) for every XDL result read within `horizon`."""
    a = asm.index(kernel + ":")
    b = asm.index(".Lfunc_end", a)
    lines = [x.split(";")[0].strip() for x in asm[a:b].split("\n")]
    ins = [x for x in lines if x and not x.startswith(".") and not x.endswith(":")]
    pairs = []
    for i, l in enumerate(ins):
        if not l.startswith("v_mfma"):
            continue
        live = _regs(_operands(l)[1][0])
        ws = 0
        for j in range(i + 1, min(len(ins), i + horizon)):
            op, ops = _operands(ins[j])
            if op in ("s_branch", "s_endpgm", "s_setpc_b64"):
                break
            # another XDL op taking the result as its accumulator is a matrix-core dependency
            # (forwarded within the XDL pipe), not a read by the vector, LDS or memory units
            if not op.startswith("v_mfma") and _reads(op, ops) & live:
                pairs.append((ws, i, j))
                break
            live -= _writes(op, ops)
            if not live:
                break
            ws += int(ops[0]) + 1 if op == "s_nop" else 1
    return pairs


def kernels(asm: str, name: str = "partials_kernel"):
    return re.findall(r"^(_ZN3fka\w*" + name + r"\w+):", asm, re.M)


def compile_asm(hipcc: str, src: str, include: str, out: str) -> str:
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", "-Xclang",
                    "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", include, "--cuda-device-only", "-S", src,
                    "-o", out], check=True, capture_output=True)
    return open(out).read()
