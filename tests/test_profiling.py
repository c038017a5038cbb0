"""Host logic of the measurement helpers: the source hash that keys the committed
HBM counters to the kernels they were taken on ignores comments and layout, and
changes with the code."""
from paper_2505_12112_amd.profiling import code_only


def test_comments_and_layout_do_not_count():
    a = 'int a; // note "x"\n/* block\n comment */ int b = \'/\';\nconst char *s = "a // b /* c */";\n'
    b = 'int a;\n\n    int b = \'/\';   // another note\nconst char *s = "a // b /* c */";'
    assert code_only(a) == code_only(b)
    assert "note" not in code_only(a) and "comment" not in code_only(a)
    assert '"a // b /* c */"' in code_only(a)  # literals are not comments


def test_code_changes_count():
    assert code_only("int a = 1; // x") != code_only("int a = 2; // x")
    assert code_only('const char *s = "a  b";') != code_only('const char *s = "a b";')
    assert code_only("x = '\\''; // q") == code_only("x =   '\\'';")
