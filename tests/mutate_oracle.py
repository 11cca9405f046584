"""Mutation sweep over the C oracle (not collected by pytest; run it by hand:
    python tests/mutate_oracle.py
). Each mutant changes one operator occurrence on one code line of oracle/rlcs_oracle.c (a sign,
a dropped factor, an index off by one, a comparison, a flag or a clip swapped); the whole pin
suite, tests/test_oracle_pins.py, runs against a copy of the oracle holding the mutant. Every
mutant the pins do not fail is printed: it is either equivalent or a gap in the pins."""
import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
src = open(f"{ROOT}/oracle/rlcs_oracle.c").read()
lines = src.split("\n")
OPS = [(r"(?<![+\-*/=<>!&|]) \+ (?!=)", " - "), (r"(?<![+\-*/=<>!&|]) - (?!=)", " + "),
       (r"gamma \* lambda", "gamma"), (r"\bt \+ 1\b", "t"), (r"\bt - 1\b", "t"),
       (r"1\.0 - ", ""), (r" >= ", " > "), (r" <= ", " < "), (r" < ", " <= "), (r" > ", " >= "),
       (r" && ", " || "), (r" \|\| ", " && "), (r"\? ([^:;]+) : ([^;]+);", r"? \2 : \1;"),
       (r"\bte\b", "tr"), (r"\bfminl?\b", "fmax"), (r"\bmin\(", "max(")]
mutants = []
in_comment = False
for i, l in enumerate(lines):
    s = l.strip()
    if s.startswith("/*") or s.startswith("*") or s.startswith("//") or s.startswith("#") or not s:
        continue
    if re.match(r"^(static |double |void |int |int64_t |const |struct |typedef )", s) and s.endswith("{"):
        continue  # signatures
    for pat, rep in OPS:
        for m in re.finditer(pat, l):
            new = l[:m.start()] + re.sub(pat, rep, l[m.start():m.end()]) + l[m.end():]
            if new != l:
                mutants.append((i, l, new))
print(len(mutants), "mutants", flush=True)

def run(k):
    i, old, new = mutants[k]
    d = os.path.join(tempfile.gettempdir(), f"msweep_{k}")
    shutil.rmtree(d, ignore_errors=True)
    shutil.copytree(f"{ROOT}/oracle", f"{d}/oracle", ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    shutil.copytree(f"{ROOT}/tests", f"{d}/tests", ignore=shutil.ignore_patterns("__pycache__"))
    shutil.copy(f"{ROOT}/workloads.py", d)
    ls = list(lines); ls[i] = new
    open(f"{d}/oracle/rlcs_oracle.c", "w").write("\n".join(ls))
    env = dict(os.environ, PYTHONPATH=d)
    try:
        r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                            f"{d}/tests/test_oracle_pins.py"], cwd=d, env=env, capture_output=True,
                           text=True, timeout=300)
        caught = r.returncode != 0
        tail = r.stdout.strip().splitlines()[-1] if r.stdout.strip() else r.stderr[-200:]
    except subprocess.TimeoutExpired:
        caught, tail = True, "timeout"
    shutil.rmtree(d, ignore_errors=True)
    return k, caught, tail

missed = []
with cf.ThreadPoolExecutor(6) as ex:
    for k, caught, tail in ex.map(run, range(len(mutants))):
        if not caught:
            i, old, new = mutants[k]
            missed.append(k)
            print(f"MISSED line {i + 1}: {old.strip()}  ->  {new.strip()}", flush=True)
print(f"caught {len(mutants) - len(missed)} of {len(mutants)}")
