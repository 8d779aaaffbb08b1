"""The oracle and the HIP path share no code, and the product never reaches the oracle."""
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def files_under(d, exts):
    for base, _, names in os.walk(os.path.join(ROOT, d)):
        for n in names:
            if n.endswith(exts):
                yield os.path.join(base, n)


def test_oracle_includes_and_imports_nothing_of_the_product():
    for f in files_under("oracle", (".c", ".h", ".py")):
        text = open(f).read()
        assert "paper_2201_01684_amd" not in text, f
        assert "gpoeo_pd.h" not in text, f
        assert not re.search(r'#include\s+"(?!oracle\.h)', text), f


def test_product_never_touches_the_oracle():
    for f in list(files_under("paper_2201_01684_amd", (".py", ".hip", ".cpp", ".h"))) + [
            os.path.join(ROOT, "include", "gpoeo_pd.h")]:
        text = open(f).read()
        assert not re.search(r"\boracle\b(?!\w)", text.replace("oracle-free", "")), f


def test_generators_hold_no_method_code():
    for f in files_under("gen", (".py",)):
        text = open(f).read()
        assert "import oracle" not in text and "paper_2201_01684_amd" not in text, f
