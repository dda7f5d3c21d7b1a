"""bench.py's kernel digest: it keys the recorded HBM counters to the code they
were taken on, so it must ignore comments and layout and see every code change."""
import bench


def test_code_only_strips_comments_keeps_strings():
    src = 'int a = 1; // note\n/* block\n comment */ const char* s = "x // y /* z */";\n\tint  b = 2;'
    assert bench.code_only(src) == 'int a = 1; const char* s = "x // y /* z */"; int b = 2;'
    assert bench.code_only("char c = '/'; // c\nint d;") == "char c = '/'; int d;"
    assert bench.code_only('const char* e = "q\\"//"; // tail') == 'const char* e = "q\\"//";'


def test_digest_ignores_comments_but_not_code():
    base = "template <int N> __device__ void f(float* x) { x[0] *= N; }\n"
    same = "// comment\ntemplate <int N>\n__device__ void f(float* x) {  /* scale */ x[0] *= N; }\n"
    other = "template <int N> __device__ void f(float* x) { x[1] *= N; }\n"
    assert bench.code_only(base) == bench.code_only(same)
    assert bench.code_only(base) != bench.code_only(other)


def test_every_kind_hashes():
    for kind in bench.DIGEST_SOURCES:
        d = bench.kernel_digest(kind)
        assert len(d) == 16 and int(d, 16) >= 0
