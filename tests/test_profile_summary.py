"""CPU: the source fingerprint that ties committed traffic measurements to
the kernel code they were taken on ignores comments and spacing only."""
from paper_2606_29223_amd.profile_summary import code_text


def test_comments_and_spacing_do_not_change_the_code_text():
    a = "int f(int x) {\n  return x + 1;   // one\n}\n"
    b = "/* header */\nint f(int x) { return x + 1; }\n"
    assert code_text(a) == code_text(b)


def test_code_and_literals_do_change_it():
    base = 'const char *s = "a // b"; int y = 2;'
    assert "a // b" in code_text(base)
    assert code_text(base) != code_text(base.replace("2", "3"))
    assert code_text("x = '/';") == "x = '/';"
    assert code_text('s = "q\\" // not a comment";') == 's = "q\\" // not a comment";'
