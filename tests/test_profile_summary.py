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


def _csv(path, header, rows):
    import csv
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


KNAME = ("void saef::(anonymous namespace)::k_compress<true>(saef::DevLayout, int, float, "
         "float, float const*, float*, float*, unsigned long*, float const*)")


def test_request_bytes_count_each_request_at_its_size(tmp_path):
    """Read bytes are 128/64/32 times the request counts, write bytes 64 times
    the 64-byte requests plus 32 times the rest; averages over dispatches."""
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    rq = tmp_path / "rq.csv"
    _csv(rq, hdr, [[1, KNAME, "TCC_EA0_RDREQ_128B_sum", 10], [1, KNAME, "TCC_EA0_RDREQ_64B_sum", 4],
                   [1, KNAME, "TCC_EA0_RDREQ_32B_sum", 2], [2, KNAME, "TCC_EA0_RDREQ_128B_sum", 30],
                   [2, KNAME, "TCC_EA0_RDREQ_64B_sum", 0], [2, KNAME, "TCC_EA0_RDREQ_32B_sum", 2]])
    wq = tmp_path / "wq.csv"
    _csv(wq, hdr, [[1, KNAME, "TCC_EA0_WRREQ_sum", 7], [1, KNAME, "TCC_EA0_WRREQ_64B_sum", 5],
                   [2, KNAME, "TCC_EA0_WRREQ_sum", 7], [2, KNAME, "TCC_EA0_WRREQ_64B_sum", 5]])
    got = P.request_bytes(P.counters_by_name(str(rq)), P.counters_by_name(str(wq)),
                          "k_compress<true>")
    assert got is not None
    rb, wb, n = got
    assert n == 2
    assert rb == 20 * 128 + 2 * 64 + 2 * 32  # averages: 20 x 128 B, 2 x 64 B, 2 x 32 B
    assert wb == 5 * 64 + 2 * 32
    assert P.request_bytes(P.counters_by_name(str(rq)), {}, "k_missing") is None


def test_timeline_prints_one_iteration(tmp_path, capsys):
    """The dispatches from the index-th marker dispatch to the next one, with
    times relative to the first."""
    hdr = ["Kernel_Name", "Queue_Id", "Grid_Size_X", "Workgroup_Size_X", "Start_Timestamp",
           "End_Timestamp"]
    step = "void saef::(anonymous namespace)::k_step<true, 1, true>(saef::DevLayout, int)"
    comp = KNAME
    rows = []
    t = 1000
    for _ in range(3):
        rows.append([step, 1, 256 * 10, 256, t, t + 300_000])
        rows.append([comp, 2, 256 * 20, 256, t + 300_000, t + 700_000])
        t += 800_000
    path = tmp_path / "trace.csv"
    _csv(path, hdr, rows)
    P.timeline(str(path), "k_step<true", 1)
    out = capsys.readouterr().out.splitlines()
    body = [line.split() for line in out[1:]]
    assert [b[0] for b in body] == ["k_step<true,", "k_compress<true>", "k_step<true,"]
    assert body[1][-3:] == ["300.0", "700.0", "400.0"]  # start, end, duration in us
