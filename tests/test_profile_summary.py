"""The measurement tooling's source hash: it names the code the counters in
profiles/ were taken on, so it changes with the code and not with comments."""
from paper_2008_05823_amd import profile_summary as P


def test_code_tokens_drop_comments_and_spacing():
    a = "int f(int x) {  // the doubled value\n  return 2 * x; /* a\n block */ }\n"
    b = "int f(int x) {\n\treturn 2 * x;\n}"
    assert P.code_tokens(a) == P.code_tokens(b) == "int f(int x) { return 2 * x; }"


def test_code_tokens_keep_code_changes():
    assert P.code_tokens("return 2 * x;") != P.code_tokens("return 3 * x;")


def test_short_kernel_names():
    name = ("void saef::(anonymous namespace)::k_compress<true>(saef::DevLayout, int, float, "
            "float, float const*, float*, float*, unsigned long*, float const*)")
    assert P.short_name(name) == "k_compress<true>"
    assert P.short_name("saef::(anonymous namespace)::k_finalize(saef::DevLayout, int, float*)") \
        == "k_finalize"
