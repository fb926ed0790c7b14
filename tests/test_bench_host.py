"""Host-side logic of bench.py (CPU only): the source fingerprint that ties a
committed traffic summary to the kernel code it was measured on."""
import bench


def test_code_text_drops_comments_and_blank_lines_only():
    src = ('int a = 1; // trailing\n'
           '/* block\n   comment */ int b = 2;\n'
           'const char *s = "x // kept /* kept */";\n'
           "char q = '\"';\n"
           '\n'
           '    // indented comment\n'
           'int c = 3;   \n')
    assert bench.code_text(src) == ('int a = 1;\n'
                                    '  int b = 2;\n'
                                    'const char *s = "x // kept /* kept */";\n'
                                    "char q = '\"';\n"
                                    'int c = 3;')


def test_source_hash_ignores_comments_but_not_code(tmp_path, monkeypatch):
    f = tmp_path / "k.hip"
    monkeypatch.setitem(bench.TRAFFIC_SOURCES, "t", [str(f)])
    f.write_text("// header\n__global__ void k(int *p) { p[0] = 1; }\n")
    h0 = bench.source_hash("t")
    f.write_text("// a longer header\n/* note */\n__global__ void k(int *p) { p[0] = 1; }  // store\n")
    assert bench.source_hash("t") == h0
    f.write_text("// header\n__global__ void k(int *p) { p[0] = 2; }\n")
    assert bench.source_hash("t") != h0
