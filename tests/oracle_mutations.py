"""Mutation check of the oracle's pins (test infrastructure; not collected by
pytest).  Each entry plants one plausible mistake in a copy of the oracle -- a
wrong constant, a swapped index or operand, a dropped term, an off-by-one in
a rounding rule -- and runs the CPU test suite on the copy; every mistake must
make at least one test fail.

    python tests/oracle_mutations.py [file-substring]   # about 30 s per mutation
"""
import os
import shutil
import subprocess
import sys
import tempfile

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTS = [
 ("oracle/philox.py", "PHILOX_W1 = 0xBB67AE85", "PHILOX_W1 = 0xBB67AE84"),
 ("oracle/philox.py", "c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0", "c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo0, hi0 ^ c3 ^ k1, lo1"),
 ("oracle/philox.py", "for r in range(PHILOX_ROUNDS):\n        if r > 0:", "for r in range(PHILOX_ROUNDS):\n        if r > 1:"),
 ("oracle/noise.py", "return r * np.cos(phi), r * np.sin(phi)", "return r * np.sin(phi), r * np.cos(phi)"),
 ("oracle/noise.py", "r = np.sqrt(-2.0 * np.log(uniform_from_word(wa)))", "r = np.sqrt(-np.log(uniform_from_word(wa)))"),
 ("oracle/noise.py", "phi = 2.0 * np.pi * angle_from_word(wb)", "phi = np.pi * angle_from_word(wb)"),
 ("oracle/noise.py", "wb = np.where(first_pair, w[1], w[3])", "wb = np.where(first_pair, w[2], w[3])"),
 ("oracle/noise.py", "return (seed & MASK32, seed >> 32)", "return (seed >> 32, seed & MASK32)"),
 ("oracle/noise.py", "return (low23(w).astype(np.float64) + 0.5) * 2.0 ** -23", "return (low23(w).astype(np.float64) + 1.0) * 2.0 ** -23"),
 ("oracle/noise.py", "return low23(w).astype(np.float64) * 2.0 ** -23", "return low23(w).astype(np.float64) * 2.0 ** -22"),
 ("oracle/noise.py", "np.uint64((1 << 23) - 1)", "np.uint64((1 << 24) - 1)"),
 ("oracle/noise.py", "phi = 2.0 * np.pi * angle_from_word(wb)", "phi = 2.0 * np.pi * uniform_from_word(wb)"),
 ("oracle/noise.py", "np.full(q.shape, tensor_id, dtype=np.uint64),\n            np.full(q.shape, domain, dtype=np.uint64))", "np.full(q.shape, domain, dtype=np.uint64),\n            np.full(q.shape, tensor_id, dtype=np.uint64))"),
 ("oracle/noise.py", "q = elems >> np.uint64(2)", "q = elems >> np.uint64(1)"),
 ("oracle/es.py", "s = np.sqrt(np.sum((r - mu) ** 2) / g)", "s = np.sqrt(np.sum((r - mu) ** 2) / (g - 1))"),
 ("oracle/es.py", "return (r - mu) / (s + _f32(eps)), 0", "return (r - mu) / s, 0"),
 ("oracle/es.py", "c = _f32(alpha) / n_members", "c = _f32(alpha)"),
 ("oracle/es.py", "c /= _f32(sigma)", "c *= _f32(sigma)"),
 ("oracle/es.py", "acc[seed] += c * int(s) * float(zi)", "acc[seed] += c * float(zi)"),
 ("oracle/es.py", "delta += wd * normals(sd, tensor_id, el)", "delta -= wd * normals(sd, tensor_id, el)"),
 ("oracle/bf16.py", "r = np.round(np.where(finite, x, 0.0) / quantum) * quantum", "r = np.floor(np.where(finite, x, 0.0) / quantum + 0.5) * quantum"),
 ("oracle/bf16.py", "quantum = np.ldexp(1.0, (lead - 7).astype(np.int32))", "quantum = np.ldexp(1.0, (lead - 8).astype(np.int32))"),
 ("oracle/es.py", "return f64_to_bf16_rne(theta + sign * _f32(sigma) * eps)", "return f64_to_bf16_rne(theta + _f32(sigma) * eps)"),
 ("oracle/es.py", "return sigma_T + (sigma0 - sigma_T) * (1.0 + np.cos(np.pi * t / T)) / 2.0", "return sigma_T + (sigma0 - sigma_T) * (1.0 + np.cos(np.pi * t / T))"),
 ("oracle/bf16.py", "x32 = x.astype(np.float32).astype(np.float64)", "x32 = x.astype(np.float64)"),
 ("oracle/bf16.py", "away = r.astype(np.float64) / 65536.0 >= 1.0 - f", "away = r.astype(np.float64) / 65536.0 > 1.0 - f"),
 ("oracle/bf16.py", "away = r.astype(np.float64) / 65536.0 >= 1.0 - f", "away = r.astype(np.float64) / 65536.0 < f"),
 ("oracle/bf16.py", "mag = np.where(away, lo + q, lo)", "mag = np.where(away, lo + q / 2, lo)"),
 ("oracle/noise.py", "    g = elems >> np.uint64(3)", "    g = elems >> np.uint64(2)"),
 ("oracle/noise.py", "word = (elems >> np.uint64(1)) & np.uint64(3)", "word = elems & np.uint64(3)"),
 ("oracle/noise.py", "shift = (elems & np.uint64(1)) * np.uint64(16)", "shift = (np.uint64(1) - (elems & np.uint64(1))) * np.uint64(16)"),
 ("oracle/noise.py", "return (picked >> np.uint64(23)).astype(np.int64)", "return (picked & np.uint64(511)).astype(np.int64)"),
 ("oracle/es.py", "mid = restore(theta_bits, seed_from, tensor_id, sign_from, sigma_from, elems=elems)", "mid = restore(theta_bits, seed_from, tensor_id, -sign_from, sigma_from, elems=elems)"),
 ("oracle/quant.py", "return scales[(elems // np.uint64(row)).astype(np.int64)]", "return scales[(elems // np.uint64(row + 8)).astype(np.int64)]"),
 ("oracle/quant.py", "ok = np.isfinite(s) & (s >= 2.0 ** -126)\n    d = sign", "ok = np.isfinite(s) & (s > 0)\n    d = sign"),
 ("oracle/quant.py", "d = sign * _f32(sigma) * normals(seed, tensor_id, el) / np.where(ok, s, 1.0)", "d = sign * _f32(sigma) * normals(seed, tensor_id, el) * np.where(ok, s, 1.0)"),
 ("oracle/quant.py", "+ (2 * r + 1) * 2.0 ** -10)", "+ r * 2.0 ** -9)"),
 ("oracle/quant.py", "+ r * 2.0 ** -16).astype(np.int64)", "+ r * 2.0 ** -17).astype(np.int64)"),
 ("oracle/quant.py", "out = np.where(ok, np.clip(q + k, -QMAX, QMAX), q)", "out = np.where(ok, np.clip(q + k, -QMAX - 1, QMAX), q)"),
 ("oracle/quant.py", "return _apply(q, -round_offset9(d, r), ok)", "return _apply(q, round_offset9(-d, r), ok)"),
 ("oracle/quant.py", "d = np.where(ok, delta / np.where(ok, s, 1.0), 0.0)", "d = np.where(ok, delta / np.where(ok, s, 1.0) / 2, 0.0)"),
 ("oracle/quant.py", "rounding_draws(round_seed, tensor_id, el, DOMAIN_ROUNDING), ok, live, 0", "rounding_draws(round_seed + 1, tensor_id, el, DOMAIN_ROUNDING), ok, live, 0"),
 ("oracle/checksum.py", "z = (z ^ (z >> np.uint64(30)))", "z = (z ^ (z >> np.uint64(31)))"),
 ("oracle/checksum.py", "MIX_M2 = 0x94D049BB133111EB", "MIX_M2 = 0x94D049BB133111EF"),
 ("oracle/checksum.py", "x = j * np.uint64(K_J) + salt + b * np.uint64(K_B)", "x = j * np.uint64(K_J) + b * np.uint64(K_B)"),
 ("oracle/checksum.py", "+ np.uint64(int(elem0) + c0)", "+ np.uint64(c0)"),
 ("oracle/checksum.py", "b = b_all[c0:c0 + chunk].astype(np.uint64)", "b = (b_all[c0:c0 + chunk] & np.uint16(0x7FFF)).astype(np.uint64)"),
 ("oracle/fp8.py", "np.exp2(e.astype(np.float64) - 7.0)", "np.exp2(e.astype(np.float64) - 8.0)"),
 ("oracle/fp8.py", "sub = m / 8.0 * 2.0 ** -6", "sub = m / 8.0 * 2.0 ** -7"),
 ("oracle/fp8.py", "(e == 15) & ((b & 7) == 7)", "(e == 15) & ((b & 7) == 6)"),
 ("oracle/fp8.py", "step = (f > u) if rule == \"restore\" else (f >= 1.0 - u)", "step = (f >= u) if rule == \"restore\" else (f >= 1.0 - u)"),
 ("oracle/fp8.py", "step = (f > u) if rule == \"restore\" else (f >= 1.0 - u)", "step = (f >= 1.0 - u)"),
 ("oracle/fp8.py", "step = (f > u) if rule == \"restore\" else (f >= 1.0 - u)", "step = (f > u) if rule == \"restore\" else (f > 1.0 - u)"),
 ("oracle/fp8.py", "u = (2 * spare_draws(seed, tensor_id, el).astype(np.float64) + 1) * 2.0 ** -10", "u = spare_draws(seed, tensor_id, el).astype(np.float64) * 2.0 ** -9"),
 ("oracle/fp8.py", "DOMAIN_ROUNDING).astype(np.float64) * 2.0 ** -16", "DOMAIN_ROUNDING).astype(np.float64) * 2.0 ** -15"),
 ("oracle/fp8.py", "out = np.where(top, E4M3_MAX, np.where(bottom, -E4M3_MAX, out))", "out = np.where(top, 416.0, np.where(bottom, -E4M3_MAX, out))"),
 ("oracle/fp8.py", "return _pass(c, round_onto_grid(_f32(v + d), \"perturb\", u), ok)", "return _pass(c, round_onto_grid(v + d, \"perturb\", u), ok)"),
 ("oracle/fp8.py", "delta = np.where(ok, delta / np.where(ok, s, 1.0), 0.0)", "delta = np.where(ok, delta * np.where(ok, s, 1.0), 0.0)"),
 ("oracle/fp8.py", "ok = np.isfinite(s) & (s >= 2.0 ** -126) & np.isfinite(v)\n    d = sign", "ok = np.isfinite(s) & (s > 0) & np.isfinite(v)\n    d = sign"),
 ("oracle/fp8.py", "return _pass(c, round_onto_grid(_f32(v - d), \"restore\", u), ok)", "return _pass(c, round_onto_grid(_f32(v + d), \"restore\", u), ok)"),
 ("oracle/es.py", "        m32 = out.astype(np.float32)", "        m32 = bf16_to_f64(f64_to_bf16_rne(out)).astype(np.float32)"),
 ("oracle/es.py", "            delta += wd * normals(sd, tensor_id, el)\n        with np.errstate(over=\"ignore\", invalid=\"ignore\"):\n            out = m + delta", "            delta += wd * normals(sd, tensor_id, el)\n        with np.errstate(over=\"ignore\", invalid=\"ignore\"):\n            out = m + delta.astype(np.float32)"),
 ("oracle/es.py", "    return m32, f64_to_bf16_rne(m32.astype(np.float64)), status", "    return m32, f64_to_bf16_rne(m), status"),
 ("oracle/es.py", "    return f64_to_bf16_rne(m + sign * _f32(sigma) * eps)", "    return f64_to_bf16_rne(m + _f32(sigma) * eps)"),

]


def _copy(tmp):
    for d in ("oracle", "tests", "paper_2608_17310_amd", "include"):
        shutil.copytree(os.path.join(REPO, d), os.path.join(tmp, d))
    for f in ("pytest.ini", "bench.py"):
        shutil.copy(os.path.join(REPO, f), tmp)


def _suite(tmp):
    # the sanitizer build checks host code, not the oracle: left out
    return subprocess.run([sys.executable, "-m", "pytest", "tests", "-q", "-x", "-m", "not gpu",
                           "-k", "not host_code", "-p", "no:cacheprovider"], cwd=tmp,
                          capture_output=True, text=True)


def main():
    only = sys.argv[1] if len(sys.argv) > 1 else ""
    muts = [m for m in MUTS if only in m[0]]
    # the unmutated copy must pass, or a failure would prove nothing
    tmp = tempfile.mkdtemp(prefix="oracle_mut_")
    try:
        _copy(tmp)
        r = _suite(tmp)
        if r.returncode != 0:
            print("the unmutated copy fails:", (r.stdout.strip().splitlines() or [""])[-1])
            return 2
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    missed = 0
    for f, a, b in muts:
        tmp = tempfile.mkdtemp(prefix="oracle_mut_")
        try:
            _copy(tmp)
            path = os.path.join(tmp, f)
            text = open(path).read()
            if a not in text:
                print("NOT APPLIED:", a)
                missed += 1
                continue
            open(path, "w").write(text.replace(a, b, 1))
            r = _suite(tmp)
            # a failed test, not a collection error, counts as caught
            caught = r.returncode == 1
            missed += not caught
            last = (r.stdout.strip().splitlines() or [""])[-1]
            print("CAUGHT " if caught else "MISSED ", b.replace("\n", " ")[:70], "|", last,
                  flush=True)
        finally:
            shutil.rmtree(tmp, ignore_errors=True)
    print(f"{len(muts)} mutations, missed: {missed}")
    return 1 if missed else 0


if __name__ == "__main__":
    sys.exit(main())
