"""Host-side logic of bench.py (CPU): the code digest that keys the committed
HBM-traffic summaries to the kernel sources they were measured on."""
import shutil

import bench


def test_code_tokens_drop_comments_only():
    src = ('int a = 1; // a comment\n/* block\n comment */ const char* s = "//kept /*kept*/";\n'
           "char q = '\\''; char r = '/';  int   b;")
    assert bench.code_tokens(src) == ('int a = 1; const char* s = "//kept /*kept*/"; '
                                      "char q = '\\''; char r = '/'; int b;")


def test_digest_ignores_comments_but_not_code(tmp_path):
    d = tmp_path / "csrc"
    shutil.copytree(bench.CSRC, d, ignore=shutil.ignore_patterns("*.o", "*.so"))
    base = bench.source_digest(str(d))
    assert base == bench.source_digest()
    f = d / "ffn.hip"
    text = f.read_text()
    f.write_text("// an added comment line\n" + text.replace("\n", "\n\n", 3))
    assert bench.source_digest(str(d)) == base
    f.write_text(text.replace("RASTER_GM", "RASTER_GM + 0", 1))
    assert bench.source_digest(str(d)) != base

