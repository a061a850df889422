"""Mutation check of the oracle's pins (run by hand, not collected by pytest):

    python tests/mutate_oracle.py [max_mutants]

Each mutant is one small edit on one code line of oracle/*.py: a comparison
flipped or loosened, +1/-1 changed, min/max or argmax/argmin swapped, a
boolean or a sign inverted, an index 0 -> 1.  It runs the CPU pin tests
(tests/test_oracle_*.py) on a copy of the repository in /tmp with the mutant
in place and reports the mutants no pin rejects.  Equivalent mutants (edits
that cannot change a result) and edits inside docstrings are among those and
are judged by reading them.
"""
import os, re, shutil, subprocess, sys, random
from concurrent.futures import ThreadPoolExecutor
SRC = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OPS = [
    (r'(?<![<>=!])<(?![<=])', '<='), (r'<=', '<'), (r'(?<![<>=!-])>(?![>=])', '>='), (r'>=', '>'),
    (r'==', '!='), (r'!=', '=='), (r'\+ 1\b', '+ 2'), (r'- 1\b', '+ 1'), (r'\bmin\(', 'max('),
    (r'\bmax\(', 'min('), (r'\bTrue\b', 'False'), (r'\bFalse\b', 'True'), (r' \+ ', ' - '),
    (r' - ', ' + '), (r'\band\b', 'or'), (r'\bor\b', 'and'), (r'\[0\]', '[1]'), (r'\[-1\]', '[0]'),
    (r'\bnot ', ''), (r' \* ', ' / '), (r'argmax\(', 'argmin('), (r'\b0\.0\b', '1.0'),
]
def sites(path):
    out = []
    lines = open(path).read().split('\n')
    in_doc = False
    for i, l in enumerate(lines):
        st = l.strip()
        if st.startswith('"""') or st.startswith("'''"):
            if not (st.count('"""') >= 2 or st.count("'''") >= 2):
                in_doc = not in_doc
            continue
        if in_doc or not st or st.startswith('#') or st.startswith('import') or st.startswith('from'):
            continue
        code = l.split('#')[0]
        for k, (pat, rep) in enumerate(OPS):
            for m in re.finditer(pat, code):
                out.append((i, m.start(), m.end(), rep, k))
    return lines, out
TESTS = sorted('tests/' + os.path.basename(f) for f in __import__('glob').glob(SRC + '/tests/test_oracle*.py'))
def run(args):
    idx, fname, line, a, b, rep = args
    d = f'/tmp/mut_{idx % 8}'
    p = os.path.join(d, 'oracle', fname)
    orig = open(os.path.join(SRC, 'oracle', fname)).read().split('\n')
    mut = list(orig); mut[line] = mut[line][:a] + rep + mut[line][b:]
    open(p, 'w').write('\n'.join(mut))
    try:
        r = subprocess.run([sys.executable, '-m', 'pytest', *TESTS, '-x', '-q', '-m', 'not gpu',
                            '-p', 'no:cacheprovider'], cwd=d, capture_output=True, text=True, timeout=120)
        assert r.returncode in (0, 1), r.stdout[-500:]
        killed = r.returncode != 0
    except subprocess.TimeoutExpired:
        killed = True
    open(p, 'w').write('\n'.join(orig))
    return (fname, line + 1, orig[line].strip(), mut[line].strip(), killed)
if __name__ == '__main__':
    import glob
    TESTS = sorted('tests/' + os.path.basename(f) for f in glob.glob(SRC + '/tests/test_oracle*.py'))
    for i in range(8):
        d = f'/tmp/mut_{i}'
        shutil.rmtree(d, ignore_errors=True)
        os.makedirs(d)
        for sub in ('oracle', 'tests', 'workloads', 'paper_2608_26112_amd'):
            shutil.copytree(os.path.join(SRC, sub), os.path.join(d, sub),
                            ignore=shutil.ignore_patterns('__pycache__', '*.so'))
    jobs = []
    for fname in sorted(os.listdir(SRC + '/oracle')):
        if not fname.endswith('.py') or fname == '__init__.py': continue
        lines, ss = sites(SRC + '/oracle/' + fname)
        for (i, a, b, rep, k) in ss:
            jobs.append((fname, i, a, b, rep))
    random.seed(1)
    if len(sys.argv) > 1: jobs = random.sample(jobs, min(len(jobs), int(sys.argv[1])))
    jobs = [(n,) + j for n, j in enumerate(jobs)]
    print('mutants', len(jobs), flush=True)
    # one worker per copy: job n runs in copy n % 8, so group by copy
    groups = [[j for j in jobs if j[0] % 8 == c] for c in range(8)]
    res = []
    def worker(g):
        return [run(j) for j in g]
    with ThreadPoolExecutor(8) as ex:
        for out in ex.map(worker, groups):
            res.extend(out)
    surv = [r for r in res if not r[4]]
    print('killed', sum(r[4] for r in res), 'survived', len(surv))
    for r in surv: print('SURV', r[0], r[1], '|', r[2], '=>', r[3])
